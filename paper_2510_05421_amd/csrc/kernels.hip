// gfx950 (CDNA4) kernels for the DVI self-speculative decode step.
//
// Every reduction here has a fixed order that depends only on the operand shape (K, head
// dim, vocabulary, chunk size), never on how many tokens are processed together.  Any
// token's result is therefore the same whether it is computed alone (one draft token),
// inside a verify block, or inside a prefill chunk: that is what makes the committed keys
// and values bitwise independent of which drafts were proposed, and the speculative output
// identical to plain greedy decoding on the same engine.
#include "kernels.h"

#include <math.h>

namespace dvi {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <DType T> struct St;
template <> struct St<DType::F32> {
    typedef float type;
    static __device__ __forceinline__ float load(const void *p, size_t i) { return ((const float *)p)[i]; }
    static __device__ __forceinline__ void store(void *p, size_t i, float v) { ((float *)p)[i] = v; }
    // D += A * B over one 1 KiB fragment pair: four 16x16x4 fp32 MFMAs, element e of each
    // lane's 16 bytes going to MFMA e (A and B use the same k assignment).
    static __device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
        return c;
    }
};
template <> struct St<DType::BF16> {
    typedef uint16_t type;
    static __device__ __forceinline__ float load(const void *p, size_t i) { return bf2f(((const uint16_t *)p)[i]); }
    static __device__ __forceinline__ void store(void *p, size_t i, float v) { ((uint16_t *)p)[i] = f2bf(v); }
    static __device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       c, 0, 0, 0);
    }
};

// Fragment-major activation layout ("FM"): the input X[M][K] of a GEMM is stored as, for each
// 16-token group g and K chunk c (KC columns), one contiguous 1 KiB block whose 16-byte lane
// slot l holds X[16g + l%16][c*KC + (l/16)*EPL .. +EPL) -- exactly the MFMA B fragment of
// lane l.  Element (m, k) of a K-column matrix therefore sits at fm_index(m, k, K).
template <DType T>
__device__ __forceinline__ size_t fm_index(int m, int k, int K) {
    constexpr int KC = (T == DType::BF16) ? 32 : 16, EPL = KC / 4;
    const int c = k / KC, rr = k - c * KC, G = rr / EPL, e = rr - G * EPL;
    return ((size_t)((m >> 4) * (K / KC) + c) * 64 + G * 16 + (m & 15)) * EPL + e;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

// Block-wide sum of 256 threads in a fixed order: butterfly inside each wave, then waves 0..3.
__device__ __forceinline__ float block_sum256(float v, float *lds4) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds4[w] = v;
    __syncthreads();
    return ((lds4[0] + lds4[1]) + lds4[2]) + lds4[3];
}
__device__ __forceinline__ float block_max256(float v, float *lds4) {
    v = wave_max(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds4[w] = v;
    __syncthreads();
    return fmaxf(fmaxf(lds4[0], lds4[1]), fmaxf(lds4[2], lds4[3]));
}

// ------------------------------------------------------------------------------------------
// weight packing
// ------------------------------------------------------------------------------------------
template <DType T>
__global__ void pack_kernel(PackSrc srcs, const int32_t *prow, int N, int K, void *dst) {
    typedef typename St<T>::type E;
    const int KC = (T == DType::BF16) ? 32 : 16, EPL = KC / 4;
    const int KT = K / KC;
    const size_t nfrag = (size_t)(N / 16) * KT * 64;
    for (size_t f = (size_t)blockIdx.x * blockDim.x + threadIdx.x; f < nfrag; f += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(f & 63);
        const size_t tile = f >> 6;
        const int nt = (int)(tile / KT), kt = (int)(tile % KT);
        const int32_t code = prow[nt * 16 + (lane & 15)];
        const E *src = (const E *)srcs.src[code >> 24] + (size_t)(code & 0xffffff) * K + kt * KC + (lane >> 4) * EPL;
        E *d = (E *)dst + f * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d[e] = src[e];
    }
}

void launch_pack(DType t, PackSrc srcs, const int32_t *prow, int N, int K, void *dst, hipStream_t s) {
    if (t == DType::BF16)
        pack_kernel<DType::BF16><<<2048, 256, 0, s>>>(srcs, prow, N, K, dst);
    else
        pack_kernel<DType::F32><<<2048, 256, 0, s>>>(srcs, prow, N, K, dst);
}

constexpr int CK = 64;  // attention key chunk (absolute positions)

// Inverse RMS of one row from its per-16-column partial sums of squares: lane l adds
// partials l, l+64, ... in order, then a butterfly, so every lane (and every workgroup that
// asks) gets the same value.
__device__ __forceinline__ float inv_rms(const float *ss, int nparts, int d, float eps) {
    const int lane = threadIdx.x & 63;
    float s = 0.f;
    for (int t = lane; t < nparts; t += 64) s += ss[t];
    s = wave_sum(s);
    return 1.0f / sqrtf(s / (float)d + eps);
}

// Sum of squares of 16 consecutive columns held as 4 values by each of the lanes
// {l, l^step, l^2step, l^3step}: ((c0-3 + c4-7) + (c8-11 + c12-15)), same tree everywhere.
__device__ __forceinline__ float sumsq16(const float v[4], int step) {
    float s = ((v[0] * v[0] + v[1] * v[1]) + v[2] * v[2]) + v[3] * v[3];
    s += __shfl_xor(s, step);
    s += __shfl_xor(s, 2 * step);
    return s;
}

// ------------------------------------------------------------------------------------------
// Skinny-M weight-streaming GEMM:  Y[m][n] = sum_k X[m][k] W[n][k],  M <= 64.
//
// One workgroup owns a band of 16 output features (one packed tile row) for all M tokens.
// Its waves split the K range into contiguous pieces (split fixed by K and the wave count,
// which depends only on N), each wave streaming 1 KiB weight fragments straight into MFMA
// A operands; tokens are the MFMA B operand (16 per group, MG groups).  The per-wave
// partial tiles are summed in wave order through LDS and the epilogue runs on wave 0.
// Output layout of a 16x16 MFMA tile: lane l holds rows 4*(l/16)+j (j = 0..3) of column
// l % 16, i.e. features nt*16 + 4*(l/16) + j of token 16*g + (l % 16).
//
// RMSNorm is folded in: when ss_in is given, X holds dtype(h * g) and row m of the result
// is scaled by 1/sqrt(mean(h[m]^2) + eps), reduced from the partial sums of squares that the
// producing epilogue wrote.  RMSNorm(h) W^T = (h*g) W^T / rms(h), so no separate pass over h.
// ------------------------------------------------------------------------------------------
// Streaming loads.  Weights are read exactly once per pass; the activation fragments are read
// once per workgroup.  Issuing both with the non-temporal hint keeps the activation reads from
// disturbing the weight stream (measured on gfx950: ordinary loads of the activations cost
// up to a third of the bandwidth at 4-16 tokens, non-temporal ones almost nothing).
__device__ __forceinline__ uint4 ld_stream(const uint4 *p) {
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    const v4u t = __builtin_nontemporal_load((const v4u *)p);
    return uint4{t.x, t.y, t.z, t.w};
}

template <DType T, int MG, int EPI, int RT, int WMAX>
__global__ void __launch_bounds__(64 * WMAX) gemm_kernel(GemmArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int nt0 = blockIdx.x * RT;
    const int KC = (T == DType::BF16) ? 32 : 16;
    const int KT = a.K / KC;
    const int c0 = (wave * KT) / nw, c1 = ((wave + 1) * KT) / nw;
    const size_t es = (T == DType::BF16) ? 2 : 4;
    const uint4 *wp = (const uint4 *)a.W + (size_t)nt0 * KT * 64 + lane;
    const size_t tile_stride = (size_t)KT * 64;

    const uint4 *xp[MG];
    bool xv[MG];
#pragma unroll
    for (int g = 0; g < MG; ++g) {
        const int m = 16 * g + (lane & 15);
        xv[g] = m < a.M;
        xp[g] = (const uint4 *)a.X + (size_t)g * KT * 64 + lane;   // FM block (g, chunk 0)
    }
    f32x4 acc[RT][MG];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int g = 0; g < MG; ++g) acc[t][g] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // Each activation fragment feeds RT weight tiles.  The loop is software-pipelined: the
    // fragments of the next U chunks are requested before the current U are multiplied, so a
    // wave always has loads in flight while its MFMAs run.
    constexpr int U = 2;
    const uint4 zero = {0u, 0u, 0u, 0u};
    uint4 w[U][RT], x[U][MG];
    auto fetch = [&](int cb, uint4 (&wf)[U][RT], uint4 (&xf)[U][MG]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = cb + u < c1;
#pragma unroll
            for (int t = 0; t < RT; ++t) wf[u][t] = in ? ld_stream(wp + t * tile_stride + (size_t)(cb + u) * 64) : zero;
#pragma unroll
            for (int g = 0; g < MG; ++g) xf[u][g] = (in && xv[g]) ? ld_stream(xp[g] + (size_t)(cb + u) * 64) : zero;
        }
    };
    fetch(c0, w, x);
    for (int c = c0; c < c1; c += U) {
        uint4 wn[U][RT], xn[U][MG];
        fetch(c + U, wn, xn);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int t = 0; t < RT; ++t)
#pragma unroll
                for (int g = 0; g < MG; ++g) acc[t][g] = St<T>::mma(w[u][t], x[u][g], acc[t][g]);
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int t = 0; t < RT; ++t) w[u][t] = wn[u][t];
#pragma unroll
            for (int g = 0; g < MG; ++g) x[u][g] = xn[u][g];
        }
    }

    // Per-wave partial tiles are summed in wave order; tile t's sum lands in wave t, which
    // then runs that tile's epilogue.
    __shared__ f32x4 red[RT][WMAX][64];
    __shared__ float sinv[64];
    if (a.ss_in != nullptr)
        for (int m = wave; m < a.M; m += nw) {
            const float v = inv_rms(a.ss_in + (size_t)m * a.ld_ss_in, a.K / 16, a.K, a.eps);
            if (lane == 0) sinv[m] = v;
        }
    f32x4 mine[MG];
#pragma unroll
    for (int g = 0; g < MG; ++g) {
#pragma unroll
        for (int t = 0; t < RT; ++t) red[t][wave][lane] = acc[t][g];
        __syncthreads();
        if (wave < RT) {
            f32x4 sum = red[wave][0][lane];
            for (int w2 = 1; w2 < nw; ++w2) sum += red[wave][w2][lane];
            mine[g] = sum;
        }
        __syncthreads();
    }
    if (wave >= RT) return;
    const int nt = nt0 + wave;

    const int G4 = lane >> 4;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
        const int m = 16 * g + (lane & 15);
        const bool valid = m < a.M;
        const float sc = (a.ss_in != nullptr && valid) ? sinv[m] : 1.0f;
        f32x4 v = mine[g];
        if (EPI == EPI_RESID) {
            float hv[4] = {0.f, 0.f, 0.f, 0.f};
            const int n0 = nt * 16 + 4 * G4;
            if (valid) {
                float *h = a.H + (size_t)m * a.ldh + n0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    hv[j] = h[j] + v[j];
                    h[j] = hv[j];
                }
            }
            const float s = sumsq16(hv, 16);
            if (valid) {
                if (a.ss_out != nullptr && G4 == 0) a.ss_out[(size_t)m * a.ld_ss_out + nt] = s;
                if (a.hg_out != nullptr)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        St<T>::store(a.hg_out, fm_index<T>(m * a.hg_rs + a.hg_off, n0 + j, a.N), hv[j] * a.g_next[n0 + j]);
            }
        } else if (EPI == EPI_QKV) {
            if (valid) {
                const int b = m / a.c, i = m - b * a.c;
                const int pos = a.lens[b] + a.pos_off + i;
                const int tiles_per_head = a.hd / 16, half = a.hd / 2;
                const int hg = nt / tiles_per_head, t = nt - hg * tiles_per_head;
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const int j = 8 * t + 2 * G4 + p;
                    float x0 = v[2 * p] * sc, x1 = v[2 * p + 1] * sc;
                    if (hg < a.n_heads + a.n_kv) {
                        const float2 cs = a.rope[(size_t)pos * half + j];
                        const float r0 = x0 * cs.x - x1 * cs.y;
                        const float r1 = x0 * cs.y + x1 * cs.x;
                        x0 = r0;
                        x1 = r1;
                    }
                    if (hg < a.n_heads) {
                        float *q = a.Q + (size_t)m * a.n_heads * a.hd + hg * a.hd;
                        q[j] = x0;
                        q[j + half] = x1;
                    } else {
                        const bool isk = hg < a.n_heads + a.n_kv;
                        const int kvh = isk ? hg - a.n_heads : hg - a.n_heads - a.n_kv;
                        void *cache = isk ? a.Kc : a.Vc;
                        const size_t base = (((size_t)b * a.n_kv + kvh) * a.s_max + pos) * a.hd;
                        St<T>::store(cache, base + j, x0);
                        St<T>::store(cache, base + j + half, x1);
                    }
                }
            }
        } else if (EPI == EPI_SWIGLU) {
            if (valid) {
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const int f = 8 * nt + 2 * G4 + p;
                    const float gt = v[2 * p] * sc, up = v[2 * p + 1] * sc;
                    const float act = gt / (1.0f + expf(-gt)) * up;
                    St<T>::store(a.A, fm_index<T>(m, f, a.N / 2), act);
                }
            }
        } else {  // EPI_LOGITS
            float best = -INFINITY;
            int bidx = 0x3fffffff, bad = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = nt * 16 + 4 * G4 + j;
                float y = v[j] * sc;
                if (a.lora_A != nullptr && valid) {
                    const float *Ar = a.lora_A + (size_t)n * a.r;
                    const float *ur = a.lora_u + (size_t)m * a.r;
                    float sacc = 0.f;
                    for (int cc = 0; cc < a.r; ++cc) sacc += Ar[cc] * ur[cc];
                    y = y + a.gamma * sacc;
                }
                if (valid) a.Z[(size_t)m * a.N + n] = y;
                if (!isfinite(y)) bad = 1;
                if (y > best) {
                    best = y;
                    bidx = n;
                }
            }
#pragma unroll
            for (int o = 16; o <= 32; o <<= 1) {
                const float ov = __shfl_xor(best, o);
                const int oi = __shfl_xor(bidx, o);
                const int ob = __shfl_xor(bad, o);
                if (ov > best || (ov == best && oi < bidx)) {
                    best = ov;
                    bidx = oi;
                }
                bad |= ob;
            }
            if (valid && G4 == 0) {
                const int nt16 = a.N / 16;
                a.part_val[(size_t)m * nt16 + nt] = best;
                a.part_idx[(size_t)m * nt16 + nt] = bidx | (bad << 30);
            }
        }
    }
}

// Launch shape of a weight matrix, a function of (N, K) only, never of M: RT 16-row tiles
// per workgroup (activations reused across them) and the K split over the workgroup's waves.
// Since neither depends on M, every output's summation order is the same for every call on
// that matrix (batch invariance).
struct GemmShape {
    int rt, waves;
};
static GemmShape gemm_shape(int N, int K, int KC, int M) {
    const int tiles = N / 16, chunks = K / KC, mg = (M + 15) / 16;
    // K split, from the matrix only: the most waves per workgroup (up to 16) that keep the whole
    // grid resident at once (8 waves per SIMD x 4 SIMDs x 256 CUs) with >= 4 chunks per wave.
    int w = 1;
    while (w < 16 && (long)tiles * (2 * w) <= 8192 && chunks / (2 * w) >= 4) w *= 2;
    // tiles per workgroup: more when there are more token groups to reuse each weight tile on
    // (16-wave workgroups have 128 registers per lane and keep one tile)
    int rt = 1;
    if (w <= 8) {
        if (mg >= 3 && tiles % 4 == 0) rt = 4;
        else if (mg >= 2 && tiles % 2 == 0) rt = 2;
        while (rt > w) rt >>= 1;
    }
    return {rt, w};
}

template <DType T, int EPI, int RT, int WMAX>
static void gemm_dispatch_mg(const GemmArgs &a, dim3 grid, dim3 block, hipStream_t s) {
    const int mg = (a.M + 15) / 16;
    switch (mg) {
        case 1: gemm_kernel<T, 1, EPI, RT, WMAX><<<grid, block, 0, s>>>(a); break;
        case 2: gemm_kernel<T, 2, EPI, RT, WMAX><<<grid, block, 0, s>>>(a); break;
        case 3: gemm_kernel<T, 3, EPI, RT, WMAX><<<grid, block, 0, s>>>(a); break;
        default: gemm_kernel<T, 4, EPI, RT, WMAX><<<grid, block, 0, s>>>(a); break;
    }
}

template <DType T, int RT, int WMAX>
static void gemm_dispatch_epi(Epi e, const GemmArgs &a, dim3 grid, dim3 block, hipStream_t s) {
    switch (e) {
        case EPI_RESID: gemm_dispatch_mg<T, EPI_RESID, RT, WMAX>(a, grid, block, s); break;
        case EPI_QKV: gemm_dispatch_mg<T, EPI_QKV, RT, WMAX>(a, grid, block, s); break;
        case EPI_SWIGLU: gemm_dispatch_mg<T, EPI_SWIGLU, RT, WMAX>(a, grid, block, s); break;
        default: gemm_dispatch_mg<T, EPI_LOGITS, RT, WMAX>(a, grid, block, s); break;
    }
}

template <DType T>
static void gemm_dispatch(Epi e, const GemmArgs &a, GemmShape sh, hipStream_t s) {
    dim3 grid(a.N / 16 / sh.rt), block(64 * sh.waves);
    if (sh.waves > 8) {
        gemm_dispatch_epi<T, 1, 16>(e, a, grid, block, s);
        return;
    }
    switch (sh.rt) {
        case 4: gemm_dispatch_epi<T, 4, 8>(e, a, grid, block, s); break;
        case 2: gemm_dispatch_epi<T, 2, 8>(e, a, grid, block, s); break;
        default: gemm_dispatch_epi<T, 1, 8>(e, a, grid, block, s); break;
    }
}

void launch_gemm(DType t, Epi e, const GemmArgs &a, hipStream_t s) {
    const GemmShape sh = gemm_shape(a.N, a.K, pack_kc(t), a.M);
    if (t == DType::BF16)
        gemm_dispatch<DType::BF16>(e, a, sh, s);
    else
        gemm_dispatch<DType::F32>(e, a, sh, s);
}

// ------------------------------------------------------------------------------------------
// Embedding gather (first layer input) and the draft-head preparation
// ------------------------------------------------------------------------------------------
// Row m = b*c + i takes token tok[b*tok_stride + i]: h = E[token] (fp32), its partial sums of
// squares per 16 columns, and hg = dtype(h * g) for the first layer's folded RMSNorm.
template <DType T>
__global__ void __launch_bounds__(256) embed_kernel(const void *emb, const int32_t *tok, int tok_stride, int c, int d,
                                                    float *h, int ldh, float *ss, int ld_ss, void *hg, const float *g) {
    const int m = blockIdx.x;
    const int b = m / c, i = m - b * c;
    const size_t row = (size_t)tok[(size_t)b * tok_stride + i] * d;
    for (int base = 0; base < d; base += 1024) {
        const int col = base + 4 * threadIdx.x;
        const bool ok = col < d;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (ok)
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = St<T>::load(emb, row + col + j);
        const float s = sumsq16(v, 1);
        if (ok) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[(size_t)m * ldh + col + j] = v[j];
                St<T>::store(hg, fm_index<T>(m, col + j, d), v[j] * g[col + j]);
            }
            if ((threadIdx.x & 3) == 0) ss[(size_t)m * ld_ss + col / 16] = s;
        }
    }
}

void launch_embed(DType t, const void *emb, const int32_t *tok, int tok_stride, int B, int c, int d, float *h, int ldh,
                  float *ss, int ld_ss, void *hg, const float *g, hipStream_t s) {
    if (t == DType::BF16)
        embed_kernel<DType::BF16><<<B * c, 256, 0, s>>>(emb, tok, tok_stride, c, d, h, ldh, ss, ld_ss, hg, g);
    else
        embed_kernel<DType::F32><<<B * c, 256, 0, s>>>(emb, tok, tok_stride, c, d, h, ldh, ss, ld_ss, hg, g);
}

// Draft head input: xhat = dtype(RMSNorm(h; g)) (the row the replay buffer logs and the head
// GEMM reads) and the LoRA projection u[c] = sum_i B_s[c][i] xhat[i].  Workgroup (c, m).
template <DType T>
__global__ void __launch_bounds__(256) head_prep_kernel(const float *h, int ldh, const float *ss, int ld_ss,
                                                        const float *g, int d, float eps, const float *Bm, int r,
                                                        void *xhat, int ldx, void *xfm, float *u) {
    __shared__ float red[4];
    const int c = blockIdx.x, m = blockIdx.y;
    const float inv = inv_rms(ss + (size_t)m * ld_ss, d / 16, d, eps);
    float acc = 0.f;
    for (int i = threadIdx.x; i < d; i += 256) {
        float x = h[(size_t)m * ldh + i] * inv * g[i];
        if (T == DType::BF16) x = bf2f(f2bf(x));
        if (c == 0) {
            St<T>::store(xhat, (size_t)m * ldx + i, x);
            St<T>::store(xfm, fm_index<T>(m, i, d), x);
        }
        acc += Bm[(size_t)c * d + i] * x;
    }
    acc = block_sum256(acc, red);
    if (threadIdx.x == 0) u[(size_t)m * r + c] = acc;
}

void launch_head_prep(DType t, const float *h, int ldh, const float *ss, int ld_ss, const float *g, int M, int d,
                      float eps, const float *Bm, int r, void *xhat, int ldx, void *xfm, float *u, hipStream_t s) {
    if (M <= 0) return;
    dim3 grid(r, M);
    if (t == DType::BF16)
        head_prep_kernel<DType::BF16><<<grid, 256, 0, s>>>(h, ldh, ss, ld_ss, g, d, eps, Bm, r, xhat, ldx, xfm, u);
    else
        head_prep_kernel<DType::F32><<<grid, 256, 0, s>>>(h, ldh, ss, ld_ss, g, d, eps, Bm, r, xhat, ldx, xfm, u);
}

// Gather rows into a compact FM buffer: dst row i = src row (i * rs + off) (FM or row-major
// source), K columns.  Used for the prefill head (last token of every sequence) and for the
// drafter update (replay rows).
template <DType T>
__global__ void __launch_bounds__(256) gather_fm_kernel(const void *src, int src_fm, int rs, int off, int K, void *dst) {
    const int i = blockIdx.x, r = i * rs + off;
    for (int k = threadIdx.x; k < K; k += 256) {
        const float v = St<T>::load(src, src_fm ? fm_index<T>(r, k, K) : (size_t)r * K + k);
        St<T>::store(dst, fm_index<T>(i, k, K), v);
    }
}

void launch_gather_fm(DType t, const void *src, bool src_fm, int rs, int off, int rows, int K, void *dst,
                      hipStream_t s) {
    if (rows <= 0) return;
    if (t == DType::BF16)
        gather_fm_kernel<DType::BF16><<<rows, 256, 0, s>>>(src, src_fm ? 1 : 0, rs, off, K, dst);
    else
        gather_fm_kernel<DType::F32><<<rows, 256, 0, s>>>(src, src_fm ? 1 : 0, rs, off, K, dst);
}

// u[m][c] = sum_i B_s[c][i] x[m][i] for already-normalised rows x.  Workgroup (c, m).
template <DType T>
__global__ void __launch_bounds__(256) lora_u_kernel(const void *x, const float *Bm, int d, int r, float *u) {
    __shared__ float red[4];
    const int c = blockIdx.x, m = blockIdx.y;
    float acc = 0.f;
    for (int i = threadIdx.x; i < d; i += 256) acc += Bm[(size_t)c * d + i] * St<T>::load(x, (size_t)m * d + i);
    acc = block_sum256(acc, red);
    if (threadIdx.x == 0) u[(size_t)m * r + c] = acc;
}

void launch_lora_u(DType t, const void *x, const float *Bm, int M, int d, int r, float *u, hipStream_t s) {
    if (M <= 0) return;
    dim3 grid(r, M);
    if (t == DType::BF16)
        lora_u_kernel<DType::BF16><<<grid, 256, 0, s>>>(x, Bm, d, r, u);
    else
        lora_u_kernel<DType::F32><<<grid, 256, 0, s>>>(x, Bm, d, r, u);
}

// ------------------------------------------------------------------------------------------
// Block-causal attention against the KV cache, split over fixed 64-position key chunks.
//
// Workgroup (chunk ch, kv head, sequence b) serves every query row of the block that reads
// this kv head (c tokens x n_heads/n_kv grouped heads); the row at position p sees keys
// 0..p.  Wave w owns keys 16w..16w+15 of the chunk: for the scores, lane l holds key
// 16w + l%16 and head-dim quarter l/16 of it in registers (a quarter-dot per lane, summed
// over the four quarters by a butterfly); for P.V, lane l holds head dims [l*HD/64, ..) of
// the wave's 16 values.  Chunk statistics are combined over the four waves in wave order.
// Keys and values are read once per workgroup straight into registers and reused by every
// row.  Each chunk's (max, sum, unnormalised output) goes to a partial slot, and
// attn_combine merges every row's chunks in chunk order.  Chunk boundaries sit at absolute
// positions, so a row's result does not depend on the other rows in its block.
// ------------------------------------------------------------------------------------------
// Load n contiguous elements (n * sizeof(E) a multiple of 16 bytes, 16-byte aligned) as floats.
template <DType T, int N>
__device__ __forceinline__ void load_row(const void *p, float *out) {
    const uint4 *q = (const uint4 *)p;
    if (T == DType::BF16) {
#pragma unroll
        for (int i = 0; i < N / 8; ++i) {
            const uint4 v = q[i];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                out[8 * i + 2 * k] = __uint_as_float(w[k] << 16);
                out[8 * i + 2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < N / 4; ++i) {
            const uint4 v = q[i];
            out[4 * i] = __uint_as_float(v.x);
            out[4 * i + 1] = __uint_as_float(v.y);
            out[4 * i + 2] = __uint_as_float(v.z);
            out[4 * i + 3] = __uint_as_float(v.w);
        }
    }
}

template <DType T, int HD>
__global__ void __launch_bounds__(256) attn_partial_kernel(AttnArgs a) {
    typedef typename St<T>::type E;
    constexpr int Q4 = HD / 4;
    constexpr int EPV = HD / 64;
    __shared__ float red_m[4], red_l[4];
    __shared__ float ow[4][HD];

    const int ch = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int len0 = a.lens[b] + a.pos_off;
    const int pmax = len0 + a.c - 1;
    const int kbase = ch * CK;
    if (kbase > pmax) return;
    const int nk = min(CK, pmax + 1 - kbase);
    const int jl = 16 * w + (lane & 15);
    const int qd = lane >> 4;
    const size_t cache0 = ((size_t)b * a.n_kv + kvh) * a.s_max + kbase;

    float kf[Q4];
    if (jl < nk) {
        load_row<T, Q4>((const E *)a.Kc + (cache0 + jl) * HD + qd * Q4, kf);
    } else {
#pragma unroll
        for (int e = 0; e < Q4; ++e) kf[e] = 0.f;
    }
    float vf[16][EPV];
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
        const int key = 16 * w + jj;
        const E *vr = (const E *)a.Vc + (cache0 + key) * HD + lane * EPV;
#pragma unroll
        for (int q = 0; q < EPV; ++q) vf[jj][q] = key < nk ? St<T>::load(vr, q) : 0.f;
    }

    const int G = a.n_heads / a.n_kv;
    const int R = a.c * G;
    for (int row = 0; row < R; ++row) {
        const int i = row / G, gi = row - i * G;
        const int h = kvh * G + gi;
        const int m = b * a.c + i;
        const int p = len0 + i;
        const int nvalid = min(nk, p + 1 - kbase);
        if (nvalid <= 0) continue;  // uniform across the workgroup
        float qv[Q4];
        load_row<DType::F32, Q4>(a.Q + (size_t)m * a.n_heads * HD + (size_t)h * HD + qd * Q4, qv);
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < Q4; ++e) dot += qv[e] * kf[e];
        dot += __shfl_xor(dot, 16);
        dot += __shfl_xor(dot, 32);
        const bool kv_ok = jl < nvalid;
        const float s = kv_ok ? dot * a.scale : -INFINITY;
        float mw = s;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) mw = fmaxf(mw, __shfl_xor(mw, o));
        if (lane == 0) red_m[w] = mw;
        __syncthreads();
        const float M = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
        const float pj = kv_ok ? expf(s - M) : 0.f;
        float lw = pj;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) lw += __shfl_xor(lw, o);
        if (lane == 0) red_l[w] = lw;
        float o[EPV];
#pragma unroll
        for (int q = 0; q < EPV; ++q) o[q] = 0.f;
        const int nkw = min(16, nvalid - 16 * w);
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) {
            const float pw = __shfl(pj, jj);
            if (jj < nkw)
#pragma unroll
                for (int q = 0; q < EPV; ++q) o[q] += pw * vf[jj][q];
        }
#pragma unroll
        for (int q = 0; q < EPV; ++q) ow[w][lane * EPV + q] = o[q];
        __syncthreads();
        if (w == 0) {
            const float L = ((red_l[0] + red_l[1]) + red_l[2]) + red_l[3];
            const size_t slot = ((size_t)m * a.n_heads + h) * a.chunk_stride + ch;
#pragma unroll
            for (int q = 0; q < EPV; ++q) {
                const int e = lane * EPV + q;
                a.part_o[slot * HD + e] = ((ow[0][e] + ow[1][e]) + ow[2][e]) + ow[3][e];
            }
            if (lane == 0) {
                a.part_ml[slot * 2 + 0] = M;
                a.part_ml[slot * 2 + 1] = L;
            }
        }
        __syncthreads();
    }
}

// Merge each row's chunk partials in chunk order: one wave per (token, head).
template <DType T, int HD>
__global__ void __launch_bounds__(256) attn_combine_kernel(AttnArgs a, int M) {
    const int lane = threadIdx.x & 63;
    const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (item >= M * a.n_heads) return;
    const int m = item / a.n_heads, h = item - m * a.n_heads;
    const int b = m / a.c, i = m - b * a.c;
    const int p = a.lens[b] + a.pos_off + i;
    const int nch = p / CK + 1;
    const size_t slot0 = ((size_t)m * a.n_heads + h) * a.chunk_stride;
    float M_ = -INFINITY;
    for (int ch = 0; ch < nch; ++ch) M_ = fmaxf(M_, a.part_ml[(slot0 + ch) * 2]);
    float L = 0.f;
    constexpr int PER = HD / 64;
    float o[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) o[q] = 0.f;
    for (int ch = 0; ch < nch; ++ch) {
        const float sc = expf(a.part_ml[(slot0 + ch) * 2] - M_);
        L += a.part_ml[(slot0 + ch) * 2 + 1] * sc;
#pragma unroll
        for (int q = 0; q < PER; ++q) o[q] += a.part_o[(slot0 + ch) * HD + lane + 64 * q] * sc;
    }
#pragma unroll
    for (int q = 0; q < PER; ++q)
        St<T>::store(a.O, fm_index<T>(m, h * HD + lane + 64 * q, a.n_heads * HD), o[q] / L);
}

template <DType T, int HD>
static void attn_launch(const AttnArgs &a, hipStream_t s) {
    dim3 grid(a.n_chunks, a.n_kv, a.B);
    attn_partial_kernel<T, HD><<<grid, 256, 0, s>>>(a);
    const int M = a.B * a.c;
    attn_combine_kernel<T, HD><<<(M * a.n_heads + 3) / 4, 256, 0, s>>>(a, M);
}

void launch_attention(DType t, const AttnArgs &a, hipStream_t s) {
    if (t == DType::BF16) {
        if (a.hd == 128) attn_launch<DType::BF16, 128>(a, s);
        else attn_launch<DType::BF16, 64>(a, s);
    } else {
        if (a.hd == 128) attn_launch<DType::F32, 128>(a, s);
        else attn_launch<DType::F32, 64>(a, s);
    }
}

// ------------------------------------------------------------------------------------------
// argmax over tile partials
// ------------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) argmax_kernel(const float *pv, const int32_t *pi, int ntiles, int32_t *out,
                                                     int out_stride, const int32_t *forced, int32_t *flags) {
    __shared__ float sv[4];
    __shared__ int si[4], sb[4];
    const int m = blockIdx.x;
    float best = -INFINITY;
    int bidx = 0x3fffffff, bad = 0;
    for (int t = threadIdx.x; t < ntiles; t += 256) {
        const float v = pv[(size_t)m * ntiles + t];
        const int code = pi[(size_t)m * ntiles + t];
        const int idx = code & 0x3fffffff;
        bad |= (code >> 30) & 1;
        if (v > best || (v == best && idx < bidx)) {
            best = v;
            bidx = idx;
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(best, o);
        const int oi = __shfl_xor(bidx, o);
        bad |= __shfl_xor(bad, o);
        if (ov > best || (ov == best && oi < bidx)) {
            best = ov;
            bidx = oi;
        }
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        sv[w] = best;
        si[w] = bidx;
        sb[w] = bad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < 4; ++k) {
            if (sv[k] > best || (sv[k] == best && si[k] < bidx)) {
                best = sv[k];
                bidx = si[k];
            }
            bad |= sb[k];
        }
        if (bidx >= 0x3fffffff) bad = 1, bidx = 0;
        out[(size_t)m * out_stride] = forced ? forced[(size_t)m * out_stride] : bidx;
        if (bad) atomicOr(flags, 1);
    }
}

void launch_argmax(const float *pv, const int32_t *pi, int M, int ntiles, int32_t *out, int out_stride,
                   const int32_t *forced, int32_t *flags, hipStream_t s) {
    if (M > 0) argmax_kernel<<<M, 256, 0, s>>>(pv, pi, ntiles, out, out_stride, forced, flags);
}

// ------------------------------------------------------------------------------------------
// Commit: longest agreeing prefix, length advance (the rollback), pending token, replay log.
// One thread does the whole (tiny) bookkeeping so ring slots are assigned in sequence order.
// ------------------------------------------------------------------------------------------
__global__ void commit_kernel(CommitArgs a) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    const int k = a.k_spec;
    int next = a.ring_state[0], valid = a.ring_state[1], cnt = 0;
    if (a.flags[0] != 0) {
        for (int b = 0; b < a.B; ++b) {
            for (int i = 0; i < k; ++i) a.tokens_out[(size_t)b * k + i] = -1;
            a.n_out[b] = 0;
            a.m_out[b] = 0;
        }
        a.copy_list[0] = 0;
        return;
    }
    for (int b = 0; b < a.B; ++b) {
        const int32_t *dr = a.drafts + (size_t)b * k;
        const int32_t *tg = a.targets + (size_t)b * k;
        int m = 0;
        while (m < k && dr[m] == tg[m]) ++m;
        const int lim = a.max_new ? max(a.max_new[b], 0) : k;
        const int n = min(min(m + 1, k), lim);
        const int prev0 = a.pending[b];
        for (int i = 0; i < k; ++i) a.tokens_out[(size_t)b * k + i] = i < n ? tg[i] : -1;
        a.lens[b] += n;
        if (n > 0) a.pending[b] = tg[n - 1];
        a.n_out[b] = n;
        a.m_out[b] = m;
        if (lim > 0 && a.ring_rows > 0) {
            const int rows = min(m + 1, k);
            for (int i = 1; i <= rows; ++i) {
                const int slot = next;
                next = (next + 1) % a.ring_rows;
                valid = min(valid + 1, a.ring_rows);
                a.ring_a[slot] = dr[i - 1];
                a.ring_r[slot] = (int8_t)(i <= m ? 1 : 0);
                a.ring_i[slot] = i;
                a.ring_prev[slot] = i == 1 ? prev0 : dr[i - 2];
                a.ring_fresh[slot] = 1;
                a.copy_list[1 + 2 * cnt] = b * k + i - 1;
                a.copy_list[2 + 2 * cnt] = slot;
                ++cnt;
            }
        }
    }
    a.copy_list[0] = cnt;
    a.ring_state[0] = next;
    a.ring_state[1] = valid;
}

void launch_commit(const CommitArgs &a, hipStream_t s) { commit_kernel<<<1, 64, 0, s>>>(a); }

__global__ void ring_copy_kernel(const int32_t *cl, const uint8_t *hk, int row_bytes, const float *vl, int V,
                                 uint8_t *rh, float *rl) {
    const int e = blockIdx.x;
    if (e >= cl[0]) return;
    const int src = cl[1 + 2 * e], slot = cl[2 + 2 * e];
    for (int k = threadIdx.x * 4; k < row_bytes; k += blockDim.x * 4)
        *(uint32_t *)(rh + (size_t)slot * row_bytes + k) = *(const uint32_t *)(hk + (size_t)src * row_bytes + k);
    for (int k = threadIdx.x; k < V; k += blockDim.x) rl[(size_t)slot * V + k] = vl[(size_t)src * V + k];
}

void launch_ring_copy(const int32_t *cl, int max_rows, const void *hk_hat, int d, int es, const float *vlogits, int V,
                      void *ring_h, float *ring_logits, hipStream_t s) {
    if (max_rows > 0)
        ring_copy_kernel<<<max_rows, 256, 0, s>>>(cl, (const uint8_t *)hk_hat, d * es, vlogits, V, (uint8_t *)ring_h,
                                                  ring_logits);
}

// ------------------------------------------------------------------------------------------
// Drafter update (Section 3.4).  Forward logits use the MFMA GEMM (EPI_LOGITS with LoRA);
// these kernels turn them into the loss gradient and the LoRA-factor gradients.
// ------------------------------------------------------------------------------------------
// stats[0] = n rows, [1] = accepted rows, [2] = fresh rows, [3] = fresh accepted rows.
__global__ void upd_counts_kernel(const int8_t *r, const int8_t *fresh, int n, float *stats) {
    if (threadIdx.x != 0) return;
    int na = 0, nf = 0, nfa = 0;
    for (int i = 0; i < n; ++i) {
        na += r[i] != 0;
        nf += fresh[i] != 0;
        nfa += (r[i] != 0) && (fresh[i] != 0);
    }
    stats[0] = (float)n;
    stats[1] = (float)na;
    stats[2] = (float)nf;
    stats[3] = (float)nfa;
}

// Row i: p = softmax(z), q = softmax(l/tau); KL, entropy, log p(a); then overwrite z with
// g = alpha p (log p - log q - KL) + beta (p - e_a) + eps p (log p + H).
__global__ void __launch_bounds__(256) upd_rows_kernel(UpdateArgs u, const float *counts) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    float *z = u.Z + (size_t)i * u.V;
    const float *lg = u.logits + (size_t)i * u.V;
    const float itau = 1.0f / u.tau;
    float mz = -INFINITY, mq = -INFINITY;
    for (int v = threadIdx.x; v < u.V; v += 256) {
        mz = fmaxf(mz, z[v]);
        mq = fmaxf(mq, lg[v] * itau);
    }
    mz = block_max256(mz, red);
    mq = block_max256(mq, red);
    float sz = 0.f, sq = 0.f;
    for (int v = threadIdx.x; v < u.V; v += 256) {
        sz += expf(z[v] - mz);
        sq += expf(lg[v] * itau - mq);
    }
    sz = block_sum256(sz, red);
    sq = block_sum256(sq, red);
    const float lz = mz + logf(sz), lq = mq + logf(sq);
    float kl = 0.f, ent = 0.f;
    for (int v = threadIdx.x; v < u.V; v += 256) {
        const float lp = z[v] - lz, lqv = lg[v] * itau - lq;
        const float p = expf(lp);
        kl += p * (lp - lqv);
        ent -= p * lp;
    }
    kl = block_sum256(kl, red);
    ent = block_sum256(ent, red);
    const int ai = u.a[i];
    const float lpa = z[ai] - lz;
    const float n = counts[0], na = counts[1], nf = counts[2];
    const float ri = (float)u.r[i], fi = (float)u.fresh[i];
    const float alpha = u.c_kl / n;
    const float beta = u.c_ce * ri / fmaxf(na, 1.f) + u.c_pg * (ri - u.baseline) * fi / fmaxf(nf, 1.f);
    const float eps = u.c_ent / n;
    __syncthreads();
    for (int v = threadIdx.x; v < u.V; v += 256) {
        const float lp = z[v] - lz, lqv = lg[v] * itau - lq;
        const float p = expf(lp);
        const float g = alpha * p * (lp - lqv - kl) + beta * (p - (v == ai ? 1.f : 0.f)) + eps * p * (lp + ent);
        z[v] = g;
    }
    if (threadIdx.x == 0) {
        float *st = u.row_stats + (size_t)i * 8;
        st[0] = kl;
        st[1] = ent;
        st[2] = lpa;
        st[3] = alpha * kl - beta * lpa - eps * ent;
    }
}

__global__ void upd_loss_kernel(UpdateArgs u, const float *counts) {
    if (threadIdx.x != 0) return;
    float loss = 0.f, kl = 0.f, ent = 0.f, ce = 0.f, pg = 0.f;
    for (int i = 0; i < u.n; ++i) {
        const float *st = u.row_stats + (size_t)i * 8;
        loss += st[3];
        kl += st[0];
        ent += st[1];
        ce -= (float)u.r[i] * st[2];
        pg -= ((float)u.r[i] - u.baseline) * (float)u.fresh[i] * st[2];
    }
    u.loss_out[0] = loss;
    u.loss_out[1] = kl / counts[0];
    u.loss_out[2] = ce / fmaxf(counts[1], 1.f);
    u.loss_out[3] = pg / fmaxf(counts[2], 1.f);
    u.loss_out[4] = ent / counts[0];
    u.loss_out[5] = counts[0];
    u.loss_out[6] = counts[1];
    u.loss_out[7] = counts[2];
    u.loss_out[8] = counts[3];
}

// dA[v][c] = gamma * sum_i g[i][v] u[i][c]   (one thread per vocabulary row v)
__global__ void __launch_bounds__(256) upd_dA_kernel(UpdateArgs u) {
    const int v = blockIdx.x * 256 + threadIdx.x;
    if (v >= u.V) return;
    float acc[64];
    for (int c = 0; c < u.rank; ++c) acc[c] = 0.f;
    for (int i = 0; i < u.n; ++i) {
        const float g = u.Z[(size_t)i * u.V + v];
        for (int c = 0; c < u.rank; ++c) acc[c] += g * u.u[(size_t)i * u.rank + c];
    }
    for (int c = 0; c < u.rank; ++c) u.dA[(size_t)v * u.rank + c] = u.gamma * acc[c];
}

// du[i][c] = gamma * sum_v A[v][c] g[i][v]   (one workgroup per row i)
__global__ void __launch_bounds__(256) upd_du_kernel(UpdateArgs u) {
    __shared__ float red[4];
    const int i = blockIdx.x;
    for (int c = 0; c < u.rank; ++c) {
        float s = 0.f;
        for (int v = threadIdx.x; v < u.V; v += 256) s += u.A[(size_t)v * u.rank + c] * u.Z[(size_t)i * u.V + v];
        s = block_sum256(s, red);
        if (threadIdx.x == 0) u.du[(size_t)i * u.rank + c] = u.gamma * s;
    }
}

// dB[c][k] = sum_i du[i][c] h[i][k]   (one thread per model dim k)
template <DType T>
__global__ void __launch_bounds__(256) upd_dB_kernel(UpdateArgs u) {
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k >= u.d) return;
    float acc[64];
    for (int c = 0; c < u.rank; ++c) acc[c] = 0.f;
    for (int i = 0; i < u.n; ++i) {
        const float hv = St<T>::load(u.Hh, (size_t)i * u.d + k);
        for (int c = 0; c < u.rank; ++c) acc[c] += u.du[(size_t)i * u.rank + c] * hv;
    }
    for (int c = 0; c < u.rank; ++c) u.dB[(size_t)c * u.d + k] = acc[c];
}

void launch_update_forward(DType t, const UpdateArgs &u, hipStream_t s) {
    float *counts = u.loss_out + 12;
    upd_counts_kernel<<<1, 64, 0, s>>>(u.r, u.fresh, u.n, counts);
    launch_lora_u(t, u.Hh, u.Bm, u.n, u.d, u.rank, u.u, s);
    const size_t es = dtype_size(t);
    for (int r0 = 0; r0 < u.n; r0 += 64) {
        const int rows = min(64, u.n - r0);
        launch_gather_fm(t, u.Hh, false, 1, r0, rows, u.d, u.xfm, s);
        GemmArgs g{};
        g.W = u.W;
        g.X = u.xfm;
        g.M = rows;
        g.N = u.V;
        g.K = u.d;
        g.Z = u.Z + (size_t)r0 * u.V;
        g.lora_A = u.A;
        g.lora_u = u.u + (size_t)r0 * u.rank;
        g.r = u.rank;
        g.gamma = u.gamma;
        g.part_val = u.part_val;
        g.part_idx = u.part_idx;
        launch_gemm(t, EPI_LOGITS, g, s);
    }
    upd_rows_kernel<<<u.n, 256, 0, s>>>(u, counts);
    upd_loss_kernel<<<1, 64, 0, s>>>(u, counts);
}

void launch_update_backward(DType t, const UpdateArgs &u, hipStream_t s) {
    (void)t;
    upd_dA_kernel<<<(u.V + 255) / 256, 256, 0, s>>>(u);
    upd_du_kernel<<<u.n, 256, 0, s>>>(u);
    if (t == DType::BF16)
        upd_dB_kernel<DType::BF16><<<(u.d + 255) / 256, 256, 0, s>>>(u);
    else
        upd_dB_kernel<DType::F32><<<(u.d + 255) / 256, 256, 0, s>>>(u);
}

__global__ void adam_kernel(float *p, const float *g, float *m, float *v, int n, float lr, float b1, float b2, float eps,
                            float c1, float c2) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.f - b1) * gi;
    const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    p[i] = p[i] - lr * (mi / c1) / (sqrtf(vi / c2) + eps);
}

void launch_adam(float *p, const float *g, float *m, float *v, int n, float lr, float b1, float b2, float eps, int step,
                 hipStream_t s) {
    const float c1 = 1.f - powf(b1, (float)step), c2 = 1.f - powf(b2, (float)step);
    adam_kernel<<<(n + 255) / 256, 256, 0, s>>>(p, g, m, v, n, lr, b1, b2, eps, c1, c2);
}

}  // namespace dvi
