// Device helpers shared by the gfx950 kernels: storage types and MFMA, the fragment-major
// activation layout, fixed-order reductions, streaming and agent-scope memory accesses, and the
// fused GEMM epilogues.
#pragma once

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

// Lane exchanges inside each row of 16 lanes by DPP (a VALU operand modifier: no LDS round trip
// and no wait, where a general shuffle goes through the LDS crossbar).  CTRL: 0xB1 = quad_perm
// (1,0,3,2), lane l reads l^1; 0x4E = quad_perm (2,3,0,1), l^2; 0x141 = half-row mirror, lane l
// reads the lane at 7 - (l%8) of its half-row; 0x140 = row mirror, 15 - (l%16) of its row.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Butterfly over each row of 16 lanes: pairs, then quads, then half-rows (the mirror pairs a lane
// with one in the other quad), then the two halves.  Every lane of a row ends with the same
// value, and it is bitwise the xor butterfly over 1, 2, 4, 8: at each level both partners hold
// the same partial, so each lane adds the same two operands in the same order (own first).
__device__ __forceinline__ float row16_sum(float v) {
    v += dpp_f32<0xB1>(v);
    v += dpp_f32<0x4E>(v);
    v += dpp_f32<0x141>(v);
    v += dpp_f32<0x140>(v);
    return v;
}
__device__ __forceinline__ float row16_max(float v) {
    v = fmaxf(v, dpp_f32<0xB1>(v));
    v = fmaxf(v, dpp_f32<0x4E>(v));
    v = fmaxf(v, dpp_f32<0x141>(v));
    v = fmaxf(v, dpp_f32<0x140>(v));
    return v;
}
// e^x as 2^(x log2 e) on the hardware exp2 (within a few ulp), for softmax weights (x <= 0;
// -inf gives 0, results below the normal range flush to 0).
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }
__device__ __forceinline__ float lane_f32(float v, int lane) {  // lane must be wave-uniform
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
// Wave reductions: each row of 16 by DPP, then the four row results read out (readlane) and
// combined as (r0 + r1) + (r2 + r3), the same tree for every lane and call.
__device__ __forceinline__ float wave_sum(float v) {
    v = row16_sum(v);
    return (lane_f32(v, 0) + lane_f32(v, 16)) + (lane_f32(v, 32) + lane_f32(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
    v = row16_max(v);
    return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
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

constexpr int CK = 64;  // attention key chunk (absolute positions)

// Inverse RMS of one row from its per-16-column partial sums of squares: lane l adds
// partials l, l+64, ... in order, then the wave sum, so every lane (and every workgroup that
// asks) gets the same value.
// inv_rms with the partial sums already in registers: v[k] holds ss[lane + 64k] (k < KP,
// nparts <= 64*KP); same summation order as inv_rms.
template <int KP>
__device__ __forceinline__ float inv_rms_regs(const float (&v)[KP], int nparts, int d, float eps) {
    const int lane = threadIdx.x & 63;
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < KP; ++k)
        if (lane + 64 * k < nparts) s += v[k];
    s = wave_sum(s);
    return 1.0f / sqrtf(s / (float)d + eps);
}

// The same as a loop, for callers short of registers.
__device__ __forceinline__ float inv_rms_loop(const float *ss, int nparts, int d, float eps) {
    const int lane = threadIdx.x & 63;
    float s = 0.f;
    for (int t = lane; t < nparts; t += 64) s += ss[t];
    s = wave_sum(s);
    return 1.0f / sqrtf(s / (float)d + eps);
}

// Up to 512 partial sums (d <= 8192) are all requested before the first add (addresses clamped
// into the row); the sum runs over lane + 64k in increasing k either way.
__device__ __forceinline__ float inv_rms(const float *ss, int nparts, int d, float eps) {
    const int lane = threadIdx.x & 63;
    constexpr int KP = 8;
    if (nparts > 64 * KP) return inv_rms_loop(ss, nparts, d, eps);
    float v[KP];
#pragma unroll
    for (int k = 0; k < KP; ++k) v[k] = ss[min(lane + 64 * k, nparts - 1)];
    return inv_rms_regs<KP>(v, nparts, d, eps);
}

// Sum of squares of 16 consecutive columns held as 4 values by each of the lanes
// {l, l^step, l^2step, l^3step}: ((c0-3 + c4-7) + (c8-11 + c12-15)), same tree everywhere.
__device__ __forceinline__ float sumsq16(const float v[4], int step) {
    float s = ((v[0] * v[0] + v[1] * v[1]) + v[2] * v[2]) + v[3] * v[3];
    s += __shfl_xor(s, step);
    s += __shfl_xor(s, 2 * step);
    return s;
}

// Streaming loads.  Weights are read exactly once per pass; the activation fragments are read
// once per workgroup.  Issuing both with the non-temporal hint keeps the activation reads from
// disturbing the weight stream (measured on gfx950: ordinary loads of the activations cost
// up to a third of the bandwidth at 4-16 tokens, non-temporal ones almost nothing).
__device__ __forceinline__ uint4 ld_stream(const uint4 *p) {
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    const v4u t = __builtin_nontemporal_load((const v4u *)p);
    return uint4{t.x, t.y, t.z, t.w};
}

// Agent-scope relaxed accesses: coherent across the L2 caches of all compute dies, no fence.
__device__ __forceinline__ void st_agent(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Coherent loads for data another workgroup wrote in the same launch: a raw buffer load with the
// sc1 cache policy reads at agent scope (never a stale L2 line), yet is an ordinary load to the
// compiler, so consecutive loads stay in flight together (agent-scope atomic loads are each
// followed by a wait for every outstanding load).  The base must be the same for every lane of
// the wave; offsets are in bytes and below 2 GiB.
constexpr int kCoherent = 16;  // sc1
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ float ld_coherent_f32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kCoherent));
}
__device__ __forceinline__ float2 ld_coherent_f32x2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    typedef unsigned v2u __attribute__((ext_vector_type(2)));
    const v2u v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCoherent);
    return float2{__uint_as_float(v.x), __uint_as_float(v.y)};
}
// Four consecutive floats in one store with the same sc1 policy (written through to where every
// XCD reads), the vector form of st_agent; ordering still comes from the release that follows.
__device__ __forceinline__ void st_coherent_f32x4(__amdgpu_buffer_rsrc_t r, uint32_t off, float a, float b, float c,
                                                  float d) {
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    const v4u v = {__float_as_uint(a), __float_as_uint(b), __float_as_uint(c), __float_as_uint(d)};
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kCoherent);
}

// Pack EPL floats into one 16-byte MFMA fragment of dtype T.
template <DType T>
__device__ __forceinline__ uint4 pack_frag(const float *v) {
    if (T == DType::BF16) {
        uint32_t w[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) w[k] = (uint32_t)f2bf(v[2 * k]) | ((uint32_t)f2bf(v[2 * k + 1]) << 16);
        return uint4{w[0], w[1], w[2], w[3]};
    }
    return uint4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
}

// Zero the elements of a 16-byte value fragment whose key index (first + e) is >= limit.
template <DType T>
__device__ __forceinline__ uint4 mask_keys(uint4 v, int first, int limit) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if (T == DType::BF16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (first + 2 * k >= limit) w[k] &= 0xffff0000u;
            if (first + 2 * k + 1 >= limit) w[k] &= 0x0000ffffu;
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (first + k >= limit) w[k] = 0u;
    }
    return uint4{w[0], w[1], w[2], w[3]};
}

// Philox4x64-10 (Salmon et al., "Parallel random numbers: as easy as 1, 2, 3", SC 2011): ten
// rounds of two 64x64 -> 128-bit products on a 4-word counter, the key advanced by the Weyl
// increments before each round after the first.
__device__ __forceinline__ void philox4x64_10(uint64_t (&c)[4], uint64_t k0, uint64_t k1) {
    constexpr uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    constexpr uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        const uint64_t hi0 = __umul64hi(M0, c[0]), lo0 = M0 * c[0];
        const uint64_t hi1 = __umul64hi(M1, c[2]), lo1 = M1 * c[2];
        const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

// Operands of a tile's epilogue that do not depend on the product (residual rows and the next
// norm's gain; positions and rotary (cos, sin)).  The epilogue wave requests them before the
// weight stream, so the epilogue after it only computes and stores.  Same lane layout as the
// epilogue: lane l, token 16*g + l%16, features nt*16 + 4*(l/16) + j.
template <int MG>
struct EpiOperands {
    float v[MG][4];  // RESID: H row values; QKV: (cos, sin) of the lane's two rotary pairs
    float g[4];      // RESID: g_next
    int pos[MG];     // QKV: position of the token
    float4 la;       // LOGITS with LoRA: float4 `lane` of the tile's A_s block (16 rows x r)
};

// The LoRA term of the logits epilogue takes A_s from registers when the rank is a multiple of
// 4 up to 16: the tile's 16 x r block is requested with the other epilogue operands, one float4
// per lane, and handed to the lanes that need it by shuffles; u (written by the kernel before)
// is read in the epilogue, all ranks at once.  Other ranks read both in the epilogue.
__device__ __forceinline__ bool lora_in_regs(const GemmArgs &a) { return a.r <= 16 && a.r % 4 == 0; }

__device__ __forceinline__ float f4_get(const float4 &v, int k) {
    return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
}

// Stage 1: everything but the rotary table, whose address needs the position.  m0: token of
// the first row group.
template <int MG, int EPI>
__device__ __forceinline__ void epilogue_prefetch(const GemmArgs &a, int nt, EpiOperands<MG> &e, int m0 = 0) {
    const int lane = threadIdx.x & 63;
    const int G4 = lane >> 4;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
        const int m = m0 + 16 * g + (lane & 15);
        const int row = m < a.M ? m : 0;  // rows past M read row 0 and are never used
        if (EPI == EPI_RESID) {
            const float4 h4 = *(const float4 *)(a.H + (size_t)row * a.ldh + nt * 16 + 4 * G4);
            e.v[g][0] = h4.x;
            e.v[g][1] = h4.y;
            e.v[g][2] = h4.z;
            e.v[g][3] = h4.w;
        } else if (EPI == EPI_QKV) {
            const int b = row / a.c, i = row - b * a.c;
            e.pos[g] = a.lens[b] + a.pos_off + i;
        }
    }
    if (EPI == EPI_RESID && a.hg_out != nullptr) {
        const float4 g4 = *(const float4 *)(a.g_next + nt * 16 + 4 * G4);
        e.g[0] = g4.x;
        e.g[1] = g4.y;
        e.g[2] = g4.z;
        e.g[3] = g4.w;
    }
    if (EPI == EPI_LOGITS && a.lora_A != nullptr && lora_in_regs(a)) {
        // the block is 16 r floats = 4 r float4s, 256-byte aligned (r % 4 == 0)
        e.la = lane < 4 * a.r ? *(const float4 *)(a.lora_A + (size_t)nt * 16 * a.r + 4 * lane)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

// Stage 2: rotary (cos, sin) at the positions of stage 1.
template <int MG, int EPI>
__device__ __forceinline__ void epilogue_prefetch_rope(const GemmArgs &a, int nt, EpiOperands<MG> &e) {
    if (EPI != EPI_QKV) return;
    const int G4 = (threadIdx.x & 63) >> 4;
    const int tiles_per_head = a.hd / 16, half = a.hd / 2;
    const int hg = nt / tiles_per_head, t = nt - hg * tiles_per_head;
    if (hg >= a.n_heads + a.n_kv) return;  // values are not rotated
#pragma unroll
    for (int g = 0; g < MG; ++g)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const float2 cs = a.rope[(size_t)e.pos[g] * half + 8 * t + 2 * G4 + p];
            e.v[g][2 * p] = cs.x;
            e.v[g][2 * p + 1] = cs.y;
        }
}

// Epilogue of one 16-feature output tile nt (rows of the weight matrix) for MG row groups of
// tokens from m0 on, run by the wave that holds the tile's reduced sums (mine[g]: MFMA output
// layout, lane l holds features nt*16 + 4*(l/16) + j of token m0 + 16*g + l%16) and the tile's
// prefetched operands e.  sinv[16*g + l%16] holds 1/rms of that token when the input was
// pre-scaled by the norm gain (folded RMSNorm).
template <DType T, int MG, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs &a, int nt, const f32x4 (&mine)[MG], const float *sinv,
                                              const EpiOperands<MG> &e, int m0 = 0) {
    const int lane = threadIdx.x & 63;
    const int G4 = lane >> 4;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
        const int m = m0 + 16 * g + (lane & 15);
        const bool valid = m < a.M;
        const float sc = (a.ss_in != nullptr && valid) ? sinv[16 * g + (lane & 15)] : 1.0f;
        f32x4 v = mine[g];
        if (EPI == EPI_RESID) {
            float hv[4] = {0.f, 0.f, 0.f, 0.f};
            const int n0 = nt * 16 + 4 * G4;
            if (valid) {
                const size_t hrow = (size_t)m * a.ldh + n0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    hv[j] = e.v[g][j] + v[j];
                    a.H[hrow + j] = hv[j];
                }
            }
            const float s = sumsq16(hv, 16);
            if (valid) {
                if (a.ss_out != nullptr && G4 == 0) a.ss_out[(size_t)m * a.ld_ss_out + nt] = s;
                if (a.hg_out != nullptr)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        St<T>::store(a.hg_out, fm_index<T>(m * a.hg_rs + a.hg_off, n0 + j, a.N), hv[j] * e.g[j]);
            }
        } else if (EPI == EPI_QKV) {
            if (valid) {
                const int b = m / a.c;
                const int pos = e.pos[g];
                const int tiles_per_head = a.hd / 16, half = a.hd / 2;
                const int hg = nt / tiles_per_head, t = nt - hg * tiles_per_head;
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const int j = 8 * t + 2 * G4 + p;
                    float x0 = v[2 * p] * sc, x1 = v[2 * p + 1] * sc;
                    if (hg < a.n_heads + a.n_kv) {
                        const float2 cs = {e.v[g][2 * p], e.v[g][2 * p + 1]};
                        const float r0 = x0 * cs.x - x1 * cs.y;
                        const float r1 = x0 * cs.y + x1 * cs.x;
                        x0 = r0;
                        x1 = r1;
                    }
                    if (hg < a.n_heads) {
                        float *q = a.Q + (size_t)m * a.n_heads * a.hd + hg * a.hd;
                        q[j] = x0;
                        q[j + half] = x1;
                    } else {  // key or value cache: the position's 64-position block, fragment-major
                        const bool key = hg < a.n_heads + a.n_kv;
                        const int kvh = hg - a.n_heads - (key ? 0 : a.n_kv), kk = pos % CK;
                        const int kc = (T == DType::BF16) ? 32 : 16;
                        const size_t blk = (((size_t)b * a.n_kv + kvh) * a.s_max + (size_t)(pos - kk)) * a.hd;
                        if (key) {
                            St<T>::store(a.Kc, blk + kv_key_offset(kc, a.hd, kk, j), x0);
                            St<T>::store(a.Kc, blk + kv_key_offset(kc, a.hd, kk, j + half), x1);
                        } else {
                            St<T>::store(a.Vc, blk + kv_val_offset(kc, a.hd, kk, j), x0);
                            St<T>::store(a.Vc, blk + kv_val_offset(kc, a.hd, kk, j + half), x1);
                        }
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
            // sampled drafting: Gumbel noise of the lane's four vocabulary entries (one block)
            float gn[4] = {0.f, 0.f, 0.f, 0.f};
            const bool sample = a.sample_tau > 0.f;
            if (sample) {
                uint64_t c[4] = {(uint64_t)(nt * 4 + G4), (uint64_t)(m * a.rng_row_stride + a.rng_row0),
                                 (uint64_t)(uint32_t)a.rng_step[0], 0ull};
                philox4x64_10(c, a.seed, 0ull);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float u = (float)(2u * (uint32_t)(c[j] >> 41) + 1u) * 0x1p-24f;
                    gn[j] = -logf(-logf(u));
                }
            }
            const bool lregs = a.lora_A != nullptr && lora_in_regs(a);
            float uv[16];
            if (lregs)
#pragma unroll
                for (int cc = 0; cc < 16; ++cc)
                    uv[cc] = (cc < a.r && valid) ? a.lora_u[(size_t)m * a.r + cc] : 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = nt * 16 + 4 * G4 + j;
                float y = v[j] * sc;
                if (lregs) {
                    // A_s[n][cc] is component cc % 4 of float4 (row * r + cc) / 4 of the block,
                    // held by that lane; the sum runs over cc in order, as below
                    const int row = 4 * G4 + j;
                    float sacc = 0.f;
#pragma unroll
                    for (int cc = 0; cc < 16; ++cc)
                        if (cc < a.r) sacc += __shfl(f4_get(e.la, cc & 3), (row * a.r + cc) >> 2) * uv[cc];
                    if (valid) y = y + a.gamma * sacc;
                } else if (a.lora_A != nullptr && valid) {
                    const float *Ar = a.lora_A + (size_t)n * a.r;
                    const float *ur = a.lora_u + (size_t)m * a.r;
                    float sacc = 0.f;
                    for (int cc = 0; cc < a.r; ++cc) sacc += Ar[cc] * ur[cc];
                    y = y + a.gamma * sacc;
                }
                if (valid) a.Z[(size_t)m * a.N + n] = y;
                if (!isfinite(y)) bad = 1;
                const float score = sample ? y / a.sample_tau + gn[j] : y;
                if (score > best) {
                    best = score;
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
            if (valid && G4 == 0 && a.part_val != nullptr) {  // argmax partials (heads only)
                const int nt16 = a.N / 16;
                a.part_val[(size_t)m * nt16 + nt] = best;
                a.part_idx[(size_t)m * nt16 + nt] = bidx | (bad << 30);
            }
        }
    }
}

}  // namespace dvi
