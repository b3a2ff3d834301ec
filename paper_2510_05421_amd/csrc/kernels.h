// Internal interface between the engine (engine.hip) and the gfx950 kernels (kernels.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dvi {

// Storage type of weights, activations fed to MFMA, and the KV cache.
enum class DType { F32 = 0, BF16 = 1 };

inline size_t dtype_size(DType t) { return t == DType::BF16 ? 2 : 4; }

// Packed weight layout ("fragment-major"): a matrix W[N][K] is cut into tiles of 16 rows x KC
// columns (KC = 32 for bf16, 16 for fp32), every tile 1 KiB.  Tile (nt, kt) sits at byte
// offset (nt * (K/KC) + kt) * 1024; inside it lane l (0..63) owns 16 contiguous bytes at 16*l:
// rows nt*16 + (l % 16), columns kt*KC + (l / 16) * EPL + [0, EPL) with EPL = KC / 4.  A wave
// streaming one 16-row band along K therefore reads consecutive 1 KiB blocks, and each lane's
// 16 bytes are directly its MFMA A-operand fragment.
inline int pack_kc(DType t) { return t == DType::BF16 ? 32 : 16; }

// KV cache layout.  Both caches hold, per (sequence, kv head), blocks of 64 positions, block c
// at element offset (c * 64) * hd of the head's region [s_max * hd].  Inside a block the
// elements are fragment-major like the weights: 1 KiB fragments whose 16 bytes per lane are an
// MFMA operand of the attention as loaded.  KC and EPL as for the weights.
//   keys   (B operand of S = Q K^T): fragment (kk / 16) * (hd / KC) + d / KC, lane
//          kk % 16 + 16 * ((d % KC) / EPL), element d % EPL;
//   values (B operand of O = P V):   fragment (d / 16) * (64 / KC) + kk / KC, lane
//          d % 16 + 16 * ((kk % KC) / EPL), element kk % EPL;
// for position kk (0..63) of the block and head dim d.  The functions give the element offset
// inside the block.
__host__ __device__ inline size_t kv_key_offset(int kc, int hd, int kk, int d) {
    const int epl = kc / 4;
    const int f = (kk / 16) * (hd / kc) + d / kc, l = kk % 16 + 16 * ((d % kc) / epl);
    return ((size_t)f * 64 + l) * epl + d % epl;
}
__host__ __device__ inline size_t kv_val_offset(int kc, int hd, int kk, int d) {
    const int epl = kc / 4;
    const int f = (d / 16) * (64 / kc) + kk / kc, l = d % 16 + 16 * ((kk % kc) / epl);
    return ((size_t)f * 64 + l) * epl + kk % epl;
}

// Rows of a packed matrix may be permuted (see the epilogues): prow[i] = src * 2^24 + row
// means packed row i is row `row` of source matrix `src` (up to three sources).
struct PackSrc {
    const void *src[3];
};
void launch_pack(DType t, PackSrc srcs, const int32_t *prow_dev, int N, int K, void *dst, hipStream_t s);

enum Epi : int {
    EPI_RESID = 0,   // H[m][n] += y                          (attention out, MLP down)
    EPI_QKV = 1,     // rotary embed q,k; q -> Q[m]; k,v -> KV cache at the token's position
    EPI_SWIGLU = 2,  // rows interleaved (gate f, up f): A[m][f] = silu(gate) * up
    EPI_LOGITS = 3,  // Z[m][n] = y (+ gamma * A_s[n] . u[m]); per-tile argmax partials
};

struct GemmArgs {
    const void *W;      // packed [N][K]
    const void *X;      // activations [M][K] (dtype of W) in fragment-major (FM) layout
    int M, N, K;
    // Folded RMSNorm: when ss_in != nullptr, X holds dtype(h * g) and output row m is scaled
    // by 1/sqrt(sum(ss_in[m][0..K/16)) / K + eps).
    const float *ss_in;
    int ld_ss_in;
    float eps;
    // token -> (sequence, block offset): m = b * c + i, position = lens[b] + pos_off + i
    int c, pos_off;
    const int32_t *lens;
    // EPI_RESID: H[m][n] += y; then per-16-column sums of squares of the new row -> ss_out,
    // and dtype(h * g_next) -> hg_out (input of the next folded RMSNorm)
    float *H;
    int ldh;
    float *ss_out;
    int ld_ss_out;
    void *hg_out;       // FM [rows][N]; token m goes to FM row m * hg_rs + hg_off
    int hg_rs, hg_off;
    const float *g_next;
    // EPI_QKV
    float *Q;           // [M][n_heads * hd] fp32
    void *Kc, *Vc;      // this layer's caches [max_batch][n_kv][s_max / 64][64-position block],
                        // blocks fragment-major (kv_key_offset, kv_val_offset)
    int n_heads, n_kv, hd, s_max;
    const float2 *rope; // [s_max][hd/2] (cos, sin)
    // EPI_SWIGLU
    void *A;            // [M][N/2] activations out (dtype, FM)
    // EPI_LOGITS
    float *Z;           // [M][N] logits
    const float *lora_A;// [N][r] or nullptr
    const float *lora_u;// [M][r]
    int r;
    float gamma;
    float *part_val;    // [M][N/16]
    int32_t *part_idx;  // [M][N/16]
    // Large-M GEMM: taken for M > 64, and for any M when large_m is set (every prefill block,
    // so a prompt's arithmetic never depends on the batch); sinv_rows is its scratch for 1/rms
    // of every token [M]
    int large_m;
    float *sinv_rows;
    // Sampled drafting (EPI_LOGITS): when sample_tau > 0 the argmax partials rank
    // z / sample_tau + g, g = -log(-log(u)), u from Philox4x64-10 with key (seed, 0) and counter
    // (n / 4, m * rng_row_stride + rng_row0, *rng_step, 0); Z keeps z itself.
    float sample_tau;
    uint64_t seed;
    const int32_t *rng_step;
    int rng_row0, rng_row_stride;
    // Decode GEMM at 33-64 tokens: when set, the K pieces run in separate workgroups that write
    // their partial tiles here (gemm_split_bytes(N, K) bytes), then a second launch adds them in
    // order and runs the epilogue; when null, one launch reduces each tile's pieces itself.
    // Either way every output gets the same arithmetic.
    float *kpart;
};
// Optional start/stop events for one launch: when set, the kernel is launched with
// hipExtLaunchKernelGGL, which stamps the events at the kernel's own start and end (the same
// interval a kernel-trace profiler reports), instead of with separate event markers.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};

// M <= 64: the weight-streaming decode GEMM.  M > 64 or large_m (prefill blocks): the large-M
// GEMM, which needs sinv_rows when ss_in is set and takes every epilogue but EPI_LOGITS
// (returns false).  Each kernel's arithmetic per output is independent of M.
bool launch_gemm(DType t, Epi e, const GemmArgs &a, hipStream_t s, const LaunchEvents &ev = {});
// Bytes of GemmArgs::kpart for an N x K matrix (64 tokens); 0 when that matrix never splits.
size_t gemm_split_bytes(DType t, int N, int K);

// Row m = b*c + i: h = E[tok[b*tok_stride + i]] (fp32, row stride ldh), its per-16-column
// sums of squares (ss, stride ld_ss) and dtype(h * g) (hg, FM, row m).
void launch_embed(DType t, const void *emb, const int32_t *tok, int tok_stride, int B, int c, int d, float *h, int ldh,
                  float *ss, int ld_ss, void *hg, const float *g, hipStream_t s);

// xhat[m] = dtype(RMSNorm(h[m]; g)) (row-major, stride ldx, and FM copy xfm) and
// u[m][c] = B_s[c] . xhat[m] (the draft head's inputs).
void launch_head_prep(DType t, const float *h, int ldh, const float *ss, int ld_ss, const float *g, int M, int d,
                      float eps, const float *Bm, int r, void *xhat, int ldx, void *xfm, float *u, hipStream_t s);

// dst (FM) row i = src row i*rs + off; src is FM when src_fm, else row-major [..][K].
void launch_gather_fm(DType t, const void *src, bool src_fm, int rs, int off, int rows, int K, void *dst,
                      hipStream_t s);

constexpr int kMaxBatch = 64;

// Rows of one prefill block that hold a sequence's last prompt token: src[b] = the row within
// the block of sequence b's last token (row b * block_len + src[b]), or -1 when that token lies in
// another block.
struct LastRows {
    int32_t src[kMaxBatch];
};
// For every sequence b with src[b] >= 0: FM row b of dst <- FM row (b * block_len + src[b]) of
// hg (K = d columns), and row b of ss_dst <- that row of ss (nps partial sums each).
void launch_gather_last(DType t, const void *hg, const float *ss, int block_len, int d, int nps, int B,
                        const LastRows &lr, void *dst, float *ss_dst, hipStream_t s);

struct AttnArgs {
    const float *Q;      // [M][n_heads*hd]
    const void *Kc;      // [max_batch][n_kv][s_max / 64][block], blocks as kv_key_offset
    const void *Vc;      // [max_batch][n_kv][s_max / 64][block], blocks as kv_val_offset
    const int32_t *lens; // [B] cache length of every sequence (device memory, so that a captured
                         // graph replays with the current lengths)
    int B, c, pos_off;
    int n_heads, n_kv, hd, s_max;
    int n_chunks;        // grid: 64-key chunks of the longest context this launch may see (an upper
                         // bound; workgroups past a sequence's own chunks exit at once)
    int chunk_stride;    // partial slots per (token, head) = ceil(s_max / 64)
    float scale;
    float *part_o;       // [M][n_heads][chunk_stride][hd]
    float *part_ml;      // [M][n_heads][chunk_stride][2]
    int32_t *counters;   // [max_batch][n_kv][kCounterStride], element 0 of each used; zero between
                         // launches (the merging workgroup resets)
    void *O;             // [M][n_heads*hd] out (dtype, FM)
    // prefill blocks: causal attention with an online softmax over each row's chunks in one kernel
    // (no partials; part_o, part_ml, counters unused)
    int flash;
};
// Merge counters sit 256 bytes apart: every chunk workgroup of a (sequence, kv head) takes its
// counter once, and counters sharing a line would serialise all heads' updates in one place.
constexpr int kCounterStride = 64;
void launch_attention(DType t, const AttnArgs &a, hipStream_t s, const LaunchEvents &ev = {});

// u[m][c] = sum_i B[c][i] * x[m][i]   (x dtype, B fp32 [r][d])
void launch_lora_u(DType t, const void *x, const float *Bm, int M, int d, int r, float *u, hipStream_t s);

// Per-row argmax over the per-tile partials (ties -> lowest id).  out[m * out_stride] =
// forced ? forced[m * out_stride] : argmax; flags[0] |= 1 on non-finite logits.
void launch_argmax(const float *part_val, const int32_t *part_idx, int M, int ntiles, int32_t *out,
                   int out_stride, const int32_t *forced, int32_t *flags, hipStream_t s);

struct CommitArgs {
    int B, k_spec;
    const int32_t *drafts;    // [B][k_spec]
    const int32_t *targets;   // [B][k_spec]
    int32_t *max_new;         // [B] or nullptr: tokens each sequence may still commit
    int max_new_dec;          // 1: subtract each sequence's n from max_new (several steps in a row)
    int32_t *lens, *pending;  // [B]
    int32_t *tokens_out;      // [B][k_spec]
    int32_t *n_out, *m_out;   // [B]
    const int32_t *flags;     // [0] != 0: non-finite logits -> commit nothing
    // replay ring
    int32_t *ring_state;      // [0] next row, [1] valid rows
    int ring_rows;
    int32_t *copy_list;       // [B*k_spec][2]: (source row b*k_spec+i-1, ring slot), count at [-1]
    int32_t *ring_a, *ring_i, *ring_prev;
    int8_t *ring_r, *ring_fresh;
    int32_t *rng_step;        // [0]: decode steps committed since the prefill (sampling counter)
};
void launch_commit(const CommitArgs &a, hipStream_t s);

// Copy the rows named by the commit's copy list into the ring (h_hat rows and verify logits).
void launch_ring_copy(const int32_t *copy_list, int max_rows, const void *hk_hat, int d, int es,
                      const float *vlogits, int V, void *ring_h, float *ring_logits, hipStream_t s);

// ---- drafter update (Section 3.4) ----
constexpr int kGradV = 128;  // vocabulary entries per workgroup of the LoRA-gradient pass
inline int grad_parts(int V) { return (V + kGradV - 1) / kGradV; }

struct UpdateArgs {
    const void *W;          // packed lm_head [V][d]
    const void *Hh;         // ring h_hat [rows][d] (dtype)
    const float *logits;    // ring logits^phi [rows][V]
    const int32_t *a;       // [rows]
    const int8_t *r, *fresh;
    int n, V, d, rank;
    float gamma, tau, baseline, c_kl, c_ce, c_pg, c_ent;
    const float *A, *Bm;    // A_s [V][r], B_s [r][d]
    float *u;               // [n][r]
    void *xfm;              // FM scratch for 256 replay rows
    float *Z;               // [n][V] drafter logits -> overwritten by g = dL/dz
    float *part_val;        // scratch for the logits GEMM epilogue
    int32_t *part_idx;
    float *row_stats;       // [n][8]
    float *dA;              // [V][r]
    float *du;              // [n][r]
    float *du_part;         // [grad_parts(V)][n][16] scratch: du shares of the vocabulary blocks
    float *dB;              // [r][d]
    float *loss_out;        // [16]: loss, kl, ce, pg, entropy, n, n_acc, n_fresh, n_fresh_acc | counts at [12..16)
};
void launch_update_forward(DType t, const UpdateArgs &u, hipStream_t s);
void launch_update_backward(DType t, const UpdateArgs &u, hipStream_t s);
void launch_adam(float *p, const float *g, float *m, float *v, int n, float lr, float b1, float b2,
                 float eps, int step, hipStream_t s);

// Streaming-read reference: every 16-byte word of buf[0, bytes) read once with the decode GEMM's
// non-temporal loads (bytes a multiple of 16); the XOR of everything read goes to sink[0] only
// when it equals a value no buffer of this library holds, so nothing is stored in practice.
void launch_stream_read(const void *buf, size_t bytes, uint32_t *sink, hipStream_t s, const LaunchEvents &ev = {});

}  // namespace dvi
