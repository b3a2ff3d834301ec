// C-ABI implementation: workspace layout, weight packing, decode-step state machine.
//
// One decode step of DVI (Section 3.3) is dvi_draft -> dvi_verify -> dvi_commit; the drafter
// update (Section 3.4) is dvi_update_drafter.  All device work is enqueued on the context's
// stream; host bookkeeping (lengths, ring occupancy) mirrors the device so capacity and state
// errors are caught before anything is launched.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <map>
#include <mutex>
#include <vector>

#include "../../include/dvi.h"
#include "kernels.h"

using namespace dvi;

namespace {

constexpr int kMaxRows = 64;   // rows of a decode-step GEMM (four 16-wide MFMA groups)
constexpr int kMaxDecodeSteps = 64;  // steps one dvi_decode_steps call may queue

enum State { S_CREATED = 0, S_READY, S_DRAFTED, S_VERIFIED };

struct LayerW {
    void *wqkv, *wo, *wgu, *wd;
    float *attn_norm, *mlp_norm;
    void *Kc, *Vc;
};

// Bump allocator over the workspace (or a size counter when base == nullptr).
struct Bump {
    uint8_t *base;
    size_t off = 0;
    explicit Bump(void *b) : base((uint8_t *)b) {}
    template <class P>
    P *take(size_t bytes) {
        off = (off + 255) & ~(size_t)255;
        P *p = base ? (P *)(base + off) : nullptr;
        off += bytes;
        return p;
    }
};

// Per-call scratch of a decode pass: attention partials (chunk_stride slots per row and head)
// and merge counters, and the vocabulary head's per-tile argmax partials.
struct Scratch {
    float *att_po = nullptr, *att_pml = nullptr;
    int32_t *att_cnt = nullptr;
    int chunk_stride = 0;
    float *part_val = nullptr;
    int32_t *part_idx = nullptr;
    float *kpart = nullptr;  // split decode GEMMs' partial tiles (null: one-launch reduction)
};

}  // namespace

struct dvi_ctx {
    dvi_config cfg;
    DType dt;
    size_t es;
    int s_cap;  // cache positions per (sequence, kv head): max_seq rounded up to a 64-key chunk
    hipStream_t stream;
    std::vector<LayerW> L;
    void *emb, *head;
    float *final_norm;
    float2 *rope;
    float *lora_A, *lora_B;
    // activations.  Residual stream h (fp32) travels with its per-16-column sums of squares
    // (ss) and dtype(h * g) for the next folded RMSNorm (hg); hk/hk_ss/hk_hg hold the k_spec
    // drafted rows of every sequence (row b*k_spec + j), which the verify then continues.
    // GEMM inputs (hg, act, attn_o, hk_hg, dfm, pfm, ufm) are in the fragment-major layout.
    float *h, *ss, *q, *hk, *hk_ss, *vlogits, *dlogits, *lora_u;
    float *sinv_rows;  // 1/rms per token for prefill-block GEMMs
    int chunk_stride = 0;  // 64-key chunks of the longest sequence (max_seq), the attention grid's cap
    void *hg, *attn_o, *act, *hk_hg, *hk_hat, *dfm, *pfm, *ufm;
    // scratch in the workspace (ws_scr), and the scratch the launches use (scr): ws_scr, except
    // inside dvi_verify_static, which points it at the library's static device array
    Scratch ws_scr, scr;
    int dev = 0;            // device current at dvi_create
    void *static_scratch = nullptr;  // that device's copy of the static array (nullptr: unresolved)
    // small device state; io block is one contiguous region copied back at commit
    int32_t *lens, *pending, *drafts, *targets, *forced, *max_new, *ids, *copy_list, *ring_state;
    int32_t *rng_step;  // [0]: decode steps committed since the prefill (the sampling counter)
    int32_t *io;  // [0,B*k) tokens | [B*k, B*k+B) n | [.., +B) m | flags[4]
    int32_t *steps_io;  // dvi_decode_steps: tokens [steps][B][k] | n [steps][B] | m [steps][B]
    int32_t *prow;
    // replay ring
    void *ring_h;
    float *ring_logits;
    int32_t *ring_a, *ring_i, *ring_prev;
    int8_t *ring_r, *ring_fresh;
    // update
    float *upd_Z, *upd_stats, *upd_dA, *upd_du, *upd_dup, *upd_dB, *upd_loss, *upd_u;
    float *mA, *vA, *mB, *vB;
    // host mirror
    int state = S_CREATED;
    int B = 0, k_spec = 0, ar_mode = 0;
    std::vector<int32_t> lens_h;
    int ring_valid_h = 0;
    bool device_error = false;
    char err[512] = {0};
    hipEvent_t ev[8];
    bool ev_ok = false;
    float ms[4] = {0, 0, 0, 0};
    int ev_pending[4] = {0, 0, 0, 0};
    // sampled drafting (0: argmax drafting)
    float samp_tau = 0.f;
    uint64_t samp_seed = 0;
    // captured decode passes: (phase, B, k_spec, variant, attention chunks) -> graph
    bool graphs = false;
    std::map<std::array<int, 5>, hipGraphExec_t> gcache;
    // kernel probe
    int probe = 0;
    std::vector<hipEvent_t> pev;
    size_t pused = 0;
    int64_t plaunch = 0;
    double pbytes = 0.0;
};

static dvi_status fail(dvi_ctx *c, dvi_status s, const char *fmt, ...) {
    if (c) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(c->err, sizeof(c->err), fmt, ap);
        va_end(ap);
        if (s == DVI_ERR_DEVICE) c->device_error = true;
    }
    return s;
}

#define HIPCHK(ctx, expr)                                                                           \
    do {                                                                                            \
        hipError_t e_ = (expr);                                                                     \
        if (e_ != hipSuccess) return fail(ctx, DVI_ERR_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
    } while (0)

#define LAUNCHCHK(ctx)                                                                              \
    do {                                                                                            \
        hipError_t e_ = hipGetLastError();                                                          \
        if (e_ != hipSuccess) return fail(ctx, DVI_ERR_DEVICE, "kernel launch: %s", hipGetErrorString(e_)); \
        if ((ctx)->device_error) return DVI_ERR_DEVICE;                                             \
    } while (0)

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

// ------------------------------------------------------------------------------------------
// Static scratch of dvi_verify_static.  The array lives in the library's device code object, so
// each GPU that loads the library holds its own copy until the process ends; host code reaches a
// device's copy only through the address hipGetSymbolAddress returns for it (the array's name is a
// host-side stand-in, not a device address).  Every context on a device shares that device's
// copy: calls that overlap on one device race on it.
// ------------------------------------------------------------------------------------------
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void *g_scratch_addr[kMaxDevices];  // per device: the address of its copy (nullptr: not resolved)

// Resolve (once per device, with that device current) the address of the device's copy.
static hipError_t resolve_static_scratch(int dev, void **out) {
    *out = nullptr;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_addr[dev] = p;
    }
    *out = g_scratch_addr[dev];
    return hipSuccess;
}

__global__ void fill_i32_kernel(int32_t *p, int n, int32_t v) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

static int qkv_rows(const dvi_config &c) { return (c.n_heads + 2 * c.n_kv_heads) * c.head_dim; }
static int cache_cap(const dvi_config &c) { return (c.max_seq + 63) / 64 * 64; }
static int m_max(const dvi_config &c) {
    int m = c.max_batch * c.max_k_spec;
    return m > kMaxRows ? m : kMaxRows;
}
// Rows of one prefill block (batch x prompt positions).  Prefill attention keeps no partials, so
// the block is bounded by its activations only.
static int prefill_rows(const dvi_config &c) {
    const int mm = m_max(c);
    return 2048 > mm ? 2048 : mm;
}
// Bytes of the split-KV attention partials of a decode step (outputs and statistics of every
// 64-key chunk of m_max rows); they are addressed with 32-bit byte offsets.
static size_t partial_bytes(const dvi_config &c) {
    return (size_t)m_max(c) * c.n_heads * (((size_t)c.max_seq + 63) / 64) * (c.head_dim + 2) * 4;
}

// Lay out (or size, when base == nullptr) everything the context keeps on the device.
static size_t layout(dvi_ctx *x, const dvi_config &c, void *base) {
    Bump b(base);
    const size_t es = c.dtype == DVI_BF16 ? 2 : 4;
    const size_t d = c.d_model, F = c.ffn_dim, V = c.vocab, qd = (size_t)c.n_heads * c.head_dim;
    const size_t kvd = (size_t)c.n_kv_heads * c.head_dim;
    const size_t M = m_max(c), Mp = prefill_rows(c), R = c.buffer_rows, r = c.lora_rank;
    const size_t cs = ((size_t)c.max_seq + 63) / 64;
    const size_t Bk = (size_t)c.max_batch * c.max_k_spec;
    const size_t cache = (size_t)c.max_batch * kvd * cache_cap(c) * es;
    std::vector<LayerW> Ls(c.n_layers);
    for (int l = 0; l < c.n_layers; ++l) {
        Ls[l].wqkv = b.take<void>((size_t)qkv_rows(c) * d * es);
        Ls[l].wo = b.take<void>(d * qd * es);
        Ls[l].wgu = b.take<void>(2 * F * d * es);
        Ls[l].wd = b.take<void>(d * F * es);
        Ls[l].attn_norm = b.take<float>(d * 4);
        Ls[l].mlp_norm = b.take<float>(d * 4);
        Ls[l].Kc = b.take<void>(cache);
        Ls[l].Vc = b.take<void>(cache);
    }
    void *emb = b.take<void>(V * d * es);
    void *head = b.take<void>(V * d * es);
    float *final_norm = b.take<float>(d * 4);
    float2 *rope = b.take<float2>((size_t)c.max_seq * (c.head_dim / 2) * 8);
    const size_t nps = d / 16;
    // activations of a GEMM call: decode steps (M rows) and prefill blocks (Mp >= M rows)
    const size_t Mp16 = (Mp + 15) / 16 * 16, Bk16 = (Bk + 15) / 16 * 16, B16 = ((size_t)c.max_batch + 15) / 16 * 16;
    float *h = b.take<float>(Mp * d * 4);
    float *ss = b.take<float>(Mp * nps * 4);
    void *hg = b.take<void>(Mp16 * d * es);
    float *q = b.take<float>(Mp * qd * 4);
    void *attn_o = b.take<void>(Mp16 * qd * es);
    void *act = b.take<void>(Mp16 * F * es);
    float *sinv_rows = b.take<float>(Mp * 4);
    float *hk = b.take<float>(Bk * d * 4);
    float *hk_ss = b.take<float>(Bk * nps * 4);
    void *hk_hg = b.take<void>(Bk16 * d * es);
    void *hk_hat = b.take<void>(Bk * d * es);
    void *dfm = b.take<void>(B16 * d * es);
    void *pfm = b.take<void>(B16 * d * es);
    void *ufm = b.take<void>((size_t)256 * d * es);
    float *vlogits = b.take<float>(M * V * 4);
    float *dlogits = b.take<float>((size_t)c.max_batch * V * 4);
    float *part_val = b.take<float>(M * (V / 16) * 4);
    int32_t *part_idx = b.take<int32_t>(M * (V / 16) * 4);
    float *lora_u = b.take<float>((M > R ? M : R) * r * 4);
    float *att_po = b.take<float>(M * c.n_heads * cs * c.head_dim * 4);
    float *att_pml = b.take<float>(M * c.n_heads * cs * 2 * 4);
    int32_t *att_cnt = b.take<int32_t>((size_t)c.max_batch * c.n_kv_heads * kCounterStride * 4);
    // partial tiles of the decode GEMMs that split their K pieces over workgroups (33-64 rows)
    size_t kpart_bytes = 0;
    if (c.max_batch * c.max_k_spec > 32 || c.max_batch > 32) {
        const DType dt = c.dtype == DVI_BF16 ? DType::BF16 : DType::F32;
        const size_t sz[] = {gemm_split_bytes(dt, qkv_rows(c), (int)d), gemm_split_bytes(dt, (int)d, (int)qd),
                             gemm_split_bytes(dt, (int)(2 * F), (int)d), gemm_split_bytes(dt, (int)d, (int)F),
                             gemm_split_bytes(dt, (int)V, (int)d)};
        for (size_t z : sz) kpart_bytes = z > kpart_bytes ? z : kpart_bytes;
    }
    float *kpart = kpart_bytes ? b.take<float>(kpart_bytes) : nullptr;
    int32_t *lens = b.take<int32_t>(c.max_batch * 4);
    int32_t *pending = b.take<int32_t>(c.max_batch * 4);
    int32_t *drafts = b.take<int32_t>(Bk * 4);
    int32_t *targets = b.take<int32_t>(Bk * 4);
    int32_t *forced = b.take<int32_t>(Bk * 4);
    int32_t *max_new = b.take<int32_t>(c.max_batch * 4);
    int32_t *ids = b.take<int32_t>((size_t)c.max_batch * c.max_seq * 4);
    int32_t *copy_list = b.take<int32_t>((1 + 2 * Bk) * 4);
    int32_t *ring_state = b.take<int32_t>(4 * 4);
    int32_t *rng_step = b.take<int32_t>(4 * 4);
    int32_t *io = b.take<int32_t>((Bk + 2 * c.max_batch + 4) * 4);
    int32_t *steps_io = b.take<int32_t>((size_t)kMaxDecodeSteps * (Bk + 2 * c.max_batch) * 4);
    size_t maxN = V;
    if ((size_t)qkv_rows(c) > maxN) maxN = qkv_rows(c);
    if (2 * F > maxN) maxN = 2 * F;
    int32_t *prow = b.take<int32_t>(maxN * 4);
    void *ring_h = b.take<void>(R * d * es);
    float *ring_logits = b.take<float>(R * V * 4);
    int32_t *ring_a = b.take<int32_t>(R * 4);
    int32_t *ring_i = b.take<int32_t>(R * 4);
    int32_t *ring_prev = b.take<int32_t>(R * 4);
    int8_t *ring_r = b.take<int8_t>(R);
    int8_t *ring_fresh = b.take<int8_t>(R);
    float *upd_Z = b.take<float>(R * V * 4);
    float *upd_stats = b.take<float>(R * 8 * 4);
    float *upd_dA = b.take<float>(V * r * 4);
    float *upd_du = b.take<float>(R * r * 4);
    float *upd_dup = b.take<float>(R * grad_parts((int)V) * 16 * 4);
    float *upd_dB = b.take<float>(r * d * 4);
    float *upd_loss = b.take<float>(16 * 4);
    float *mA = b.take<float>(V * r * 4);
    float *vA = b.take<float>(V * r * 4);
    float *mB = b.take<float>(r * d * 4);
    float *vB = b.take<float>(r * d * 4);
    if (x && base) {
        x->L = Ls;
        x->emb = emb; x->head = head; x->final_norm = final_norm; x->rope = rope;
        x->h = h; x->ss = ss; x->hg = hg; x->q = q; x->attn_o = attn_o; x->act = act; x->sinv_rows = sinv_rows;
        x->hk = hk; x->hk_ss = hk_ss; x->hk_hg = hk_hg; x->hk_hat = hk_hat;
        x->dfm = dfm; x->pfm = pfm; x->ufm = ufm;
        x->vlogits = vlogits; x->dlogits = dlogits;
        x->lora_u = lora_u;
        x->ws_scr.att_po = att_po; x->ws_scr.att_pml = att_pml; x->ws_scr.att_cnt = att_cnt;
        x->ws_scr.chunk_stride = (int)cs; x->ws_scr.part_val = part_val; x->ws_scr.part_idx = part_idx;
        x->ws_scr.kpart = kpart;
        x->scr = x->ws_scr;
        x->chunk_stride = (int)cs;
        x->lens = lens; x->pending = pending; x->drafts = drafts; x->targets = targets; x->forced = forced;
        x->max_new = max_new; x->ids = ids; x->copy_list = copy_list; x->ring_state = ring_state; x->rng_step = rng_step; x->io = io;
        x->steps_io = steps_io;
        x->prow = prow;
        x->ring_h = ring_h; x->ring_logits = ring_logits; x->ring_a = ring_a; x->ring_i = ring_i;
        x->ring_prev = ring_prev; x->ring_r = ring_r; x->ring_fresh = ring_fresh;
        x->upd_Z = upd_Z; x->upd_stats = upd_stats; x->upd_dA = upd_dA; x->upd_du = upd_du; x->upd_dup = upd_dup; x->upd_dB = upd_dB;
        x->upd_loss = upd_loss; x->upd_u = lora_u;
        x->mA = mA; x->vA = vA; x->mB = mB; x->vB = vB;
    }
    return align_up(b.off);
}

static const char *check_config(const dvi_config *c) {
    if (!c) return "null config";
    if (c->dtype != DVI_FP32 && c->dtype != DVI_BF16) return "dtype must be DVI_FP32 or DVI_BF16";
    const int kc = c->dtype == DVI_BF16 ? 32 : 16;
    if (c->n_layers < 1) return "n_layers < 1";
    if (c->split_k < 1 || c->split_k > c->n_layers) return "split_k must be in [1, n_layers]";
    if (c->d_model <= 0 || c->d_model % kc) return "d_model must be a positive multiple of 32 (bf16) / 16 (fp32)";
    if (c->d_model > 8192) return "d_model must be <= 8192";
    if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
    if (c->n_heads < 1 || c->n_kv_heads < 1 || c->n_heads % c->n_kv_heads) return "n_heads must be a multiple of n_kv_heads";
    if ((c->n_heads * c->head_dim) % kc) return "n_heads*head_dim not a multiple of the K chunk";
    if (c->ffn_dim <= 0 || c->ffn_dim % kc || c->ffn_dim % 8) return "ffn_dim must be a positive multiple of 32 (bf16) / 16 (fp32)";
    if (c->vocab <= 0 || c->vocab % 16) return "vocab must be a positive multiple of 16";
    if (c->max_batch < 1 || c->max_k_spec < 1 || c->max_k_spec > 16) return "max_batch >= 1, 1 <= max_k_spec <= 16";
    if (c->max_batch * c->max_k_spec > kMaxRows) return "max_batch * max_k_spec must be <= 64";
    if (c->max_batch > dvi::kMaxBatch) return "max_batch must be <= 64";
    if (c->max_seq < 2) return "max_seq < 2";
    if (partial_bytes(*c) >= ((size_t)2 << 30)) return "max_seq too long: the attention partials of 64 rows must stay under 2 GiB";
    if (c->lora_rank < 1 || c->lora_rank > 64) return "lora_rank must be in [1, 64]";
    if (c->buffer_rows < 1) return "buffer_rows < 1";
    if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f)) return "rms_eps and rope_theta must be > 0";
    return nullptr;
}

extern "C" size_t dvi_workspace_bytes(const dvi_config *cfg) {
    if (check_config(cfg)) return 0;
    return layout(nullptr, *cfg, nullptr);
}

static dvi_status to_f32_vec(dvi_ctx *x, const void *src_dev, size_t n, float *dst_dev) {
    std::vector<uint8_t> tmp(n * x->es);
    std::vector<float> f(n);
    HIPCHK(x, hipMemcpy(tmp.data(), src_dev, n * x->es, hipMemcpyDeviceToHost));
    for (size_t i = 0; i < n; ++i) {
        if (x->dt == DType::BF16) {
            uint32_t u = (uint32_t)((uint16_t *)tmp.data())[i] << 16;
            memcpy(&f[i], &u, 4);
        } else {
            f[i] = ((float *)tmp.data())[i];
        }
    }
    HIPCHK(x, hipMemcpy(dst_dev, f.data(), n * 4, hipMemcpyHostToDevice));
    return DVI_OK;
}

static dvi_status pack(dvi_ctx *x, PackSrc s, const std::vector<int32_t> &prow, int N, int K, void *dst) {
    HIPCHK(x, hipMemcpy(x->prow, prow.data(), prow.size() * 4, hipMemcpyHostToDevice));
    launch_pack(x->dt, s, x->prow, N, K, dst, x->stream);
    LAUNCHCHK(x);
    HIPCHK(x, hipStreamSynchronize(x->stream));
    return DVI_OK;
}

static inline int32_t code(int src, int row) { return (src << 24) | row; }

extern "C" dvi_status dvi_create(const dvi_config *cfg, const dvi_weights *w, void *ws, size_t ws_bytes, void *stream,
                                 dvi_ctx **out) {
    if (!out) return DVI_ERR_ARG;
    *out = nullptr;
    const char *why = check_config(cfg);
    if (why) return DVI_ERR_ARG;
    if (!w || !ws) return DVI_ERR_ARG;
    if (((uintptr_t)ws) & 255) return DVI_ERR_ARG;
    const size_t need = layout(nullptr, *cfg, nullptr);
    if (ws_bytes < need) return DVI_ERR_CAPACITY;
    dvi_ctx *x = new dvi_ctx();
    x->cfg = *cfg;
    x->dt = cfg->dtype == DVI_BF16 ? DType::BF16 : DType::F32;
    x->es = dtype_size(x->dt);
    x->s_cap = cache_cap(*cfg);
    x->stream = (hipStream_t)stream;
    x->graphs = stream != nullptr;
    layout(x, *cfg, ws);
    // the static scratch of dvi_verify_static on this device (a failure only disables that call)
    if (hipGetDevice(&x->dev) == hipSuccess && resolve_static_scratch(x->dev, &x->static_scratch) != hipSuccess)
        x->static_scratch = nullptr;
    (void)hipGetLastError();
    x->lora_A = w->lora_A;
    x->lora_B = w->lora_B;
    const dvi_config &c = *cfg;
    const int d = c.d_model, F = c.ffn_dim, V = c.vocab, hd = c.head_dim, H = c.n_heads, Hkv = c.n_kv_heads;
    dvi_status st;
#define TRY(e)                            \
    do {                                  \
        st = (e);                         \
        if (st != DVI_OK) {               \
            *out = x;                     \
            return st;                    \
        }                                 \
    } while (0)
    // Row orders.  QKV: inside every head, packed local row 4g+2p+s (g = 0..3, p, s = 0..1) of
    // tile t is head dim j + s*hd/2 with j = 8t + 2g + p, so an MFMA lane holds both members of
    // two rotary pairs.  Gate/up: local row 4g+2p+s of tile t is feature 8t+2g+p of the gate
    // (s = 0) or up (s = 1) projection, so a lane holds (gate, up) of two features.
    std::vector<int32_t> pq(qkv_rows(c)), pgu(2 * F), pid_d(d), pid_v(V);
    for (int i = 0; i < qkv_rows(c); ++i) {
        const int hg = i / hd, loc = i % hd, t = loc / 16, lr = loc % 16;
        const int g = lr / 4, p = (lr % 4) / 2, s = lr % 2;
        const int dim = 8 * t + 2 * g + p + s * (hd / 2);
        if (hg < H) pq[i] = code(0, hg * hd + dim);
        else if (hg < H + Hkv) pq[i] = code(1, (hg - H) * hd + dim);
        else pq[i] = code(2, (hg - H - Hkv) * hd + dim);
    }
    for (int i = 0; i < 2 * F; ++i) {
        const int t = i / 16, lr = i % 16, g = lr / 4, p = (lr % 4) / 2, s = lr % 2;
        pgu[i] = code(s, 8 * t + 2 * g + p);
    }
    for (int i = 0; i < d; ++i) pid_d[i] = code(0, i);
    for (int i = 0; i < V; ++i) pid_v[i] = code(0, i);
    for (int l = 0; l < c.n_layers; ++l) {
        PackSrc s{};
        s.src[0] = w->wq[l]; s.src[1] = w->wk[l]; s.src[2] = w->wv[l];
        TRY(pack(x, s, pq, qkv_rows(c), d, x->L[l].wqkv));
        s.src[0] = w->wo[l];
        TRY(pack(x, s, pid_d, d, H * hd, x->L[l].wo));
        s.src[0] = w->w_gate[l]; s.src[1] = w->w_up[l];
        TRY(pack(x, s, pgu, 2 * F, d, x->L[l].wgu));
        s.src[0] = w->w_down[l];
        TRY(pack(x, s, pid_d, d, F, x->L[l].wd));
        TRY(to_f32_vec(x, w->attn_norm[l], d, x->L[l].attn_norm));
        TRY(to_f32_vec(x, w->mlp_norm[l], d, x->L[l].mlp_norm));
    }
    {
        PackSrc s{};
        s.src[0] = w->lm_head;
        TRY(pack(x, s, pid_v, V, d, x->head));
    }
    TRY(to_f32_vec(x, w->final_norm, d, x->final_norm));
    if (hipMemcpy(x->emb, w->tok_emb, (size_t)V * d * x->es, hipMemcpyDeviceToDevice) != hipSuccess) {
        *out = x;
        return fail(x, DVI_ERR_DEVICE, "embedding copy failed");
    }
    // Rotary table: entry (p, j) = (cos, sin) of p * theta^(-2j/hd), computed in double.
    {
        std::vector<float> rt((size_t)c.max_seq * (hd / 2) * 2);
        for (int p = 0; p < c.max_seq; ++p)
            for (int j = 0; j < hd / 2; ++j) {
                const double ang = (double)p * pow((double)c.rope_theta, -2.0 * j / (double)hd);
                rt[((size_t)p * (hd / 2) + j) * 2 + 0] = (float)cos(ang);
                rt[((size_t)p * (hd / 2) + j) * 2 + 1] = (float)sin(ang);
            }
        if (hipMemcpy(x->rope, rt.data(), rt.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
            *out = x;
            return fail(x, DVI_ERR_DEVICE, "rope upload failed");
        }
    }
    // Zero the small state, ring and optimiser moments.
    {
        const size_t Bk = (size_t)c.max_batch * c.max_k_spec;
        const size_t R = c.buffer_rows, r = c.lora_rank;
        struct Z { void *p; size_t n; } zs[] = {
            {x->lens, (size_t)c.max_batch * 4}, {x->pending, (size_t)c.max_batch * 4}, {x->drafts, Bk * 4},
            {x->targets, Bk * 4}, {x->io, (Bk + 2 * (size_t)c.max_batch + 4) * 4}, {x->ring_state, 16}, {x->rng_step, 16},
            {x->ring_fresh, R}, {x->ring_r, R}, {x->mA, (size_t)V * r * 4}, {x->vA, (size_t)V * r * 4},
            {x->mB, r * d * 4}, {x->vB, r * d * 4}, {x->ws_scr.att_cnt, (size_t)c.max_batch * c.n_kv_heads * kCounterStride * 4}};
        for (const Z &z : zs)
            if (hipMemset(z.p, 0, z.n) != hipSuccess) {
                *out = x;
                return fail(x, DVI_ERR_DEVICE, "zero-fill failed");
            }
        if (hipDeviceSynchronize() != hipSuccess) {
            *out = x;
            return fail(x, DVI_ERR_DEVICE, "zero-fill failed");
        }
    }
#undef TRY
    x->ev_ok = true;
    for (int i = 0; i < 8; ++i)
        if (hipEventCreate(&x->ev[i]) != hipSuccess) x->ev_ok = false;
    x->lens_h.assign(c.max_batch, 0);
    x->state = S_CREATED;
    *out = x;
    return DVI_OK;
}

static void drop_graphs(dvi_ctx *x) {
    for (auto &kv : x->gcache) (void)hipGraphExecDestroy(kv.second);
    x->gcache.clear();
}

extern "C" void dvi_destroy(dvi_ctx *x) {
    if (!x) return;
    drop_graphs(x);
    if (x->ev_ok)
        for (int i = 0; i < 8; ++i) (void)hipEventDestroy(x->ev[i]);
    for (auto &e : x->pev) (void)hipEventDestroy(e);
    delete x;
}

extern "C" const char *dvi_last_error(const dvi_ctx *x) { return x ? x->err : "null context"; }

// ------------------------------------------------------------------------------------------
// forward pieces
// ------------------------------------------------------------------------------------------
constexpr size_t kProbeMax = 8192;

// The probed kernel class is launched with a start/stop event pair that the launch itself
// stamps at the kernel's start and end.
static LaunchEvents probe_begin(dvi_ctx *x, int cls) {
    LaunchEvents ev;
    if (x->probe == cls && x->pused + 2 <= x->pev.size()) {
        ev.start = x->pev[x->pused];
        ev.stop = x->pev[x->pused + 1];
    }
    return ev;
}
static void probe_end(dvi_ctx *x, const LaunchEvents &ev, double bytes) {
    if (!ev.start) return;
    x->pused += 2;
    x->plaunch += 1;
    x->pbytes += bytes;
}

// Algorithmic bytes of one GEMM launch: the weight matrix once, activations in, results out.
static double gemm_bytes(const dvi_ctx *x, Epi e, int M, int N, int K) {
    const double es = (double)x->es;
    double b = (double)N * K * es + (double)M * K * es;
    const dvi_config &c = x->cfg;
    switch (e) {
        case EPI_RESID: b += 2.0 * M * N * 4; break;                               // h read + written
        case EPI_QKV: b += (double)M * c.n_heads * c.head_dim * 4 + 2.0 * M * c.n_kv_heads * c.head_dim * es; break;
        case EPI_SWIGLU: b += (double)M * (N / 2) * es; break;
        case EPI_LOGITS: b += (double)M * N * 4; break;
    }
    return b;
}

static void gemm(dvi_ctx *x, Epi e, int cls, const void *W, const void *X, int M, int N, int K, GemmArgs a) {
    a.W = W;
    a.X = X;
    a.M = M;
    a.N = N;
    a.K = K;
    a.sinv_rows = x->sinv_rows;
    a.kpart = x->scr.kpart;
    const LaunchEvents ev = probe_begin(x, cls);
    if (!launch_gemm(x->dt, e, a, x->stream, ev))
        (void)fail(x, DVI_ERR_DEVICE, "no GEMM variant for %d rows of epilogue %d", M, (int)e);
    probe_end(x, ev, gemm_bytes(x, e, M, N, K));
}

// Layers [l0, l1) on M = B*c rows; row r = b*c+i sits at position lens[b] + pos_off + i.  The
// fp32 residual stream and its sums of squares live at row r*rs of h / ss.  hg (FM, compact rows
// r) holds dtype(h * attn_norm[l0]) on entry; the last layer's MLP-down epilogue writes
// dtype(h * g) for the norm that follows layer l1-1 (attn_norm[l1], or final_norm at L) to FM row
// r*out_rs + out_off of out_hg.
static const float *next_gain(dvi_ctx *x, int l) {
    return l + 1 < x->cfg.n_layers ? x->L[l + 1].attn_norm : x->final_norm;
}

// Attention grid of a call whose rows reach at most position pmax: its 64-key chunks rounded up
// to a multiple of 4 (a 256-position bucket), so that a captured pass stays valid until the
// longest sequence crosses a bucket edge.  Workgroups past a sequence's own chunks exit at once.
constexpr int kSampleRowStride = 16;  // counter row = sequence * 16 + draft index (k_spec <= 16)

static int attn_chunks(const dvi_ctx *x, int pmax) {
    const int n = (pmax / 64 + 1 + 3) / 4 * 4;
    return n < x->chunk_stride ? n : x->chunk_stride;
}

static int max_len(const dvi_ctx *x) {
    int m = 0;
    for (int b = 0; b < x->B; ++b) m = x->lens_h[b] > m ? x->lens_h[b] : m;
    return m;
}

static dvi_status run_layers(dvi_ctx *x, int l0, int l1, int B, int c, int pos_off, int n_chunks, float *h, float *ss,
                             void *hg, int rs, void *out_hg, int out_rs, int out_off, bool prefill = false) {
    const dvi_config &cf = x->cfg;
    const int d = cf.d_model, F = cf.ffn_dim, H = cf.n_heads, Hkv = cf.n_kv_heads, hd = cf.head_dim;
    const int nps = d / 16;
    const int M = B * c;
    for (int l = l0; l < l1; ++l) {
        const LayerW &Lw = x->L[l];
        GemmArgs a{};
        a.large_m = prefill;
        a.ss_in = ss;
        a.ld_ss_in = rs * nps;
        a.eps = cf.rms_eps;
        a.c = c;
        a.pos_off = pos_off;
        a.lens = x->lens;
        a.Q = x->q;
        a.Kc = Lw.Kc;
        a.Vc = Lw.Vc;
        a.n_heads = H;
        a.n_kv = Hkv;
        a.hd = hd;
        a.s_max = x->s_cap;
        a.rope = x->rope;
        gemm(x, EPI_QKV, DVI_PROBE_QKV, Lw.wqkv, hg, M, qkv_rows(cf), d, a);
        AttnArgs at{};
        at.Q = x->q;
        at.Kc = Lw.Kc;
        at.Vc = Lw.Vc;
        at.lens = x->lens;
        at.B = B;
        at.c = c;
        at.pos_off = pos_off;
        at.n_heads = H;
        at.n_kv = Hkv;
        at.hd = hd;
        at.s_max = x->s_cap;
        at.scale = 1.0f / sqrtf((float)hd);
        at.n_chunks = n_chunks;
        at.chunk_stride = x->scr.chunk_stride;
        at.part_o = x->scr.att_po;
        at.part_ml = x->scr.att_pml;
        at.counters = x->scr.att_cnt;
        at.O = x->attn_o;
        at.flash = prefill ? 1 : 0;
        const LaunchEvents ev = probe_begin(x, DVI_PROBE_ATTENTION);
        launch_attention(x->dt, at, x->stream, ev);
        if (ev.start) {
            // keys and values of positions 0..p read once per (sequence, kv head); q in, o out
            double kv = 0.0;
            for (int b = 0; b < B; ++b) kv += (double)(x->lens_h[b] + pos_off + c) * Hkv * hd * 2.0 * x->es;
            probe_end(x, ev, kv + (double)M * H * hd * (4.0 + x->es));
        }
        GemmArgs r{};
        r.large_m = prefill;
        r.H = h;
        r.ldh = rs * d;
        r.ss_out = ss;
        r.ld_ss_out = rs * nps;
        r.hg_out = hg;
        r.hg_rs = 1;
        r.hg_off = 0;
        r.g_next = Lw.mlp_norm;
        gemm(x, EPI_RESID, DVI_PROBE_ATTN_OUT, Lw.wo, x->attn_o, M, d, H * hd, r);
        GemmArgs g{};
        g.large_m = prefill;
        g.ss_in = ss;
        g.ld_ss_in = rs * nps;
        g.eps = cf.rms_eps;
        g.A = x->act;
        gemm(x, EPI_SWIGLU, DVI_PROBE_GATE_UP, Lw.wgu, hg, M, 2 * F, d, g);
        r.g_next = next_gain(x, l);
        if (l == l1 - 1) {
            r.hg_out = out_hg;
            r.hg_rs = out_rs;
            r.hg_off = out_off;
        }
        gemm(x, EPI_RESID, DVI_PROBE_DOWN, Lw.wd, x->act, M, d, F, r);
    }
    LAUNCHCHK(x);
    return DVI_OK;
}

// io block: tokens [max_batch*max_k_spec] | n [max_batch] | m [max_batch] | flags [4]
static int io_n(const dvi_ctx *x) { return x->cfg.max_batch * x->cfg.max_k_spec; }
static int io_m(const dvi_ctx *x) { return io_n(x) + x->cfg.max_batch; }
static int io_flags(const dvi_ctx *x) { return io_m(x) + x->cfg.max_batch; }
static int io_words(const dvi_ctx *x) { return io_flags(x) + 4; }
static int32_t *flags_ptr(dvi_ctx *x) { return x->io + io_flags(x); }

// Vocabulary head on M rows of X (FM): logits -> Z, argmax -> out (stride).
// ss_in != nullptr: X holds dtype(h * final_norm) and rows are scaled by 1/rms (folded norm).
// draft_j >= 0: the draft head of draft index j, sampled when sampling is on.
static void head(dvi_ctx *x, const void *X, const float *ss_in, int ld_ss, int M, float *Z, bool lora, int32_t *out,
                 int out_stride, const int32_t *forced, int draft_j = -1) {
    const dvi_config &cf = x->cfg;
    GemmArgs a{};
    if (draft_j >= 0 && x->samp_tau > 0.f) {
        a.sample_tau = x->samp_tau;
        a.seed = x->samp_seed;
        a.rng_step = x->rng_step;
        a.rng_row0 = draft_j;
        a.rng_row_stride = kSampleRowStride;
    }
    a.ss_in = ss_in;
    a.ld_ss_in = ld_ss;
    a.eps = cf.rms_eps;
    a.Z = Z;
    a.part_val = x->scr.part_val;
    a.part_idx = x->scr.part_idx;
    if (lora) {
        a.lora_A = x->lora_A;
        a.lora_u = x->lora_u;
        a.r = cf.lora_rank;
        a.gamma = cf.lora_gamma;
    }
    gemm(x, EPI_LOGITS, DVI_PROBE_HEAD, x->head, X, M, cf.vocab, cf.d_model, a);
    launch_argmax(x->scr.part_val, x->scr.part_idx, M, cf.vocab / 16, out, out_stride, forced, flags_ptr(x), x->stream);
}

static void ev_begin(dvi_ctx *x, int phase) {
    if (x->ev_ok) (void)hipEventRecord(x->ev[2 * phase], x->stream);
}
static void ev_end(dvi_ctx *x, int phase) {
    if (x->ev_ok) {
        (void)hipEventRecord(x->ev[2 * phase + 1], x->stream);
        x->ev_pending[phase] = 1;
    }
}

// Runs body (a sequence of kernel launches on the context's stream) directly, or as the captured
// graph of key, capturing it on first use.  A failed capture leaves nothing cached.
constexpr size_t kMaxGraphs = 64;

template <typename Body>
static dvi_status run_pass(dvi_ctx *x, const std::array<int, 5> &key, Body &&body) {
    if (!x->graphs || x->probe != DVI_PROBE_OFF) return body();
    auto it = x->gcache.find(key);
    if (it == x->gcache.end()) {
        if (x->gcache.size() >= kMaxGraphs) drop_graphs(x);
        HIPCHK(x, hipStreamBeginCapture(x->stream, hipStreamCaptureModeThreadLocal));
        const dvi_status st = body();
        hipGraph_t g = nullptr;
        const hipError_t e = hipStreamEndCapture(x->stream, &g);
        if (st != DVI_OK) {
            if (g) (void)hipGraphDestroy(g);
            return st;
        }
        if (e != hipSuccess) return fail(x, DVI_ERR_DEVICE, "hipStreamEndCapture: %s", hipGetErrorString(e));
        hipGraphExec_t ge = nullptr;
        const hipError_t ei = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
        (void)hipGraphDestroy(g);
        if (ei != hipSuccess) return fail(x, DVI_ERR_DEVICE, "hipGraphInstantiate: %s", hipGetErrorString(ei));
        it = x->gcache.emplace(key, ge).first;
    }
    HIPCHK(x, hipGraphLaunch(it->second, x->stream));
    return DVI_OK;
}

extern "C" dvi_status dvi_set_sampling(dvi_ctx *x, float tau, uint64_t seed) {
    if (!x) return DVI_ERR_ARG;
    if (!(tau >= 0.f) || !isfinite(tau)) return fail(x, DVI_ERR_ARG, "sampling temperature must be finite and >= 0");
    if (x->state == S_DRAFTED || x->state == S_VERIFIED) return fail(x, DVI_ERR_STATE, "sampling set during a step");
    x->samp_tau = tau;
    x->samp_seed = seed;
    drop_graphs(x);  // the draft head's arguments changed
    return DVI_OK;
}

extern "C" dvi_status dvi_set_graphs(dvi_ctx *x, int32_t enable) {
    if (!x) return DVI_ERR_ARG;
    if (enable && x->stream == nullptr) return fail(x, DVI_ERR_ARG, "graphs need a stream other than the null stream");
    if (!enable) drop_graphs(x);
    x->graphs = enable != 0;
    return DVI_OK;
}

// ------------------------------------------------------------------------------------------
// C ABI: decode step
// ------------------------------------------------------------------------------------------
extern "C" dvi_status dvi_prefill(dvi_ctx *x, int32_t batch, const int32_t *ids, const int32_t *lens, int32_t stride,
                                  int32_t *first_tok) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state == S_DRAFTED || x->state == S_VERIFIED) return fail(x, DVI_ERR_STATE, "prefill during a step");
    const dvi_config &cf = x->cfg;
    if (!ids || !lens || !first_tok) return fail(x, DVI_ERR_ARG, "null argument");
    if (batch < 1) return fail(x, DVI_ERR_ARG, "batch < 1");
    if (batch > cf.max_batch) return fail(x, DVI_ERR_CAPACITY, "batch %d > max_batch %d", batch, cf.max_batch);
    // Prompts may differ in length: every sequence runs over P = the longest prompt, the shorter
    // ones padded with token 0 at the end.  A row attends only to positions at or before its own,
    // so padding changes no real row; its keys and values lie past the sequence's length, where
    // decoding overwrites them before any row can read them.
    int P = 0;
    for (int b = 0; b < batch; ++b) {
        if (lens[b] < 1 || lens[b] > stride) return fail(x, DVI_ERR_ARG, "prompt length %d of sequence %d outside [1, stride]", lens[b], b);
        if (lens[b] + 1 > cf.max_seq)
            return fail(x, DVI_ERR_CAPACITY, "prompt length %d leaves no room in max_seq %d", lens[b], cf.max_seq);
        P = lens[b] > P ? lens[b] : P;
    }
    std::vector<int32_t> packed((size_t)batch * P, 0);
    for (int b = 0; b < batch; ++b)
        for (int i = 0; i < lens[b]; ++i) {
            const int32_t t = ids[(size_t)b * stride + i];
            if (t < 0 || t >= cf.vocab) return fail(x, DVI_ERR_ARG, "token id %d out of range", t);
            packed[(size_t)b * P + i] = t;
        }
    const int d = cf.d_model;
    HIPCHK(x, hipMemcpyAsync(x->ids, packed.data(), packed.size() * 4, hipMemcpyHostToDevice, x->stream));
    HIPCHK(x, hipMemsetAsync(x->lens, 0, cf.max_batch * 4, x->stream));
    HIPCHK(x, hipMemsetAsync(x->rng_step, 0, 4, x->stream));
    HIPCHK(x, hipMemsetAsync(flags_ptr(x), 0, 16, x->stream));
    x->B = batch;
    for (int b = 0; b < cf.max_batch; ++b) x->lens_h[b] = 0;
    const int c = (prefill_rows(cf) / batch) < 1 ? 1 : prefill_rows(cf) / batch;  // positions per block
    const int nps = d / 16;
    for (int s0 = 0; s0 < P; s0 += c) {
        const int cc = (P - s0) < c ? P - s0 : c;
        launch_embed(x->dt, x->emb, x->ids + s0, P, batch, cc, d, x->h, d, x->ss, nps, x->hg, x->L[0].attn_norm,
                     x->stream);
        dvi_status st =
            run_layers(x, 0, cf.n_layers, batch, cc, s0, attn_chunks(x, s0 + cc - 1), x->h, x->ss, x->hg, 1, x->hg, 1, 0,
                       true);
        if (st != DVI_OK) return st;
        // each sequence's last prompt token -> its first generated token: collect the head's
        // input rows (pfm, with their sums of squares in hk_ss) from the block that holds them
        LastRows lr;
        bool any = false;
        for (int b = 0; b < kMaxBatch; ++b) {
            const int i = b < batch ? lens[b] - 1 - s0 : -1;
            lr.src[b] = (i >= 0 && i < cc) ? i : -1;
            any = any || lr.src[b] >= 0;
        }
        if (any) launch_gather_last(x->dt, x->hg, x->ss, cc, d, nps, batch, lr, x->pfm, x->hk_ss, x->stream);
    }
    head(x, x->pfm, x->hk_ss, nps, batch, x->vlogits, false, x->pending, 1, nullptr);
    std::vector<int32_t> lh(cf.max_batch, 0);
    for (int b = 0; b < batch; ++b) lh[b] = lens[b];
    HIPCHK(x, hipMemcpyAsync(x->lens, lh.data(), cf.max_batch * 4, hipMemcpyHostToDevice, x->stream));
    int32_t fl[4];
    HIPCHK(x, hipMemcpyAsync(first_tok, x->pending, batch * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipMemcpyAsync(fl, flags_ptr(x), 16, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    LAUNCHCHK(x);
    for (int b = 0; b < batch; ++b) x->lens_h[b] = lens[b];
    x->k_spec = 1;  // dvi_read_logits now returns the prefill's head logits, one row per sequence
    x->state = S_READY;
    if (fl[0]) return fail(x, DVI_ERR_NUMERIC, "non-finite logits in prefill");
    return DVI_OK;
}

// One draft pass (Section 3.3): k_spec serial single-token passes of layers 1..k from the
// pending tokens, each followed by the draft head (or, in plain decoding, by nothing).
static dvi_status draft_pass(dvi_ctx *x, int k_spec, bool forced, int nck) {
    const dvi_config &cf = x->cfg;
    const int B = x->B, d = cf.d_model, nps = d / 16;
    x->ar_mode = (k_spec == 1 && !forced) ? 1 : 0;
    const dvi_status st = run_pass(x, {0, B, k_spec, x->ar_mode + 2 * (forced ? 1 : 0), nck}, [&]() -> dvi_status {
        for (int j = 0; j < k_spec; ++j) {
            // draft token j of sequence b lives in row b*k_spec + j of hk / hk_ss / hk_hg
            const int32_t *tok = j == 0 ? x->pending : x->drafts + (j - 1);
            float *h = x->hk + (size_t)j * d;
            float *ss = x->hk_ss + (size_t)j * nps;
            launch_embed(x->dt, x->emb, tok, j == 0 ? 1 : k_spec, B, 1, d, h, k_spec * d, ss, k_spec * nps, x->hg,
                         x->L[0].attn_norm, x->stream);
            // the last draft layer hands its rows to the verify: FM row b*k_spec + j of hk_hg
            dvi_status sl = run_layers(x, 0, cf.split_k, B, 1, j, nck, h, ss, x->hg, k_spec, x->hk_hg, k_spec, j);
            if (sl != DVI_OK) return sl;
            if (!x->ar_mode) {
                void *xh = (uint8_t *)x->hk_hat + (size_t)j * d * x->es;
                launch_head_prep(x->dt, h, k_spec * d, ss, k_spec * nps, x->final_norm, B, d, cf.rms_eps, x->lora_B,
                                 cf.lora_rank, xh, k_spec * d, x->dfm, x->lora_u, x->stream);
                head(x, x->dfm, nullptr, 0, B, x->dlogits, true, x->drafts + j, k_spec,
                     forced ? x->forced + j : nullptr, j);
            }
        }
        LAUNCHCHK(x);
        return DVI_OK;
    });
    if (st != DVI_OK) return st;
    if (x->ar_mode) HIPCHK(x, hipMemsetAsync(x->drafts, 0xff, (size_t)B * 4, x->stream));
    LAUNCHCHK(x);
    x->k_spec = k_spec;
    return DVI_OK;
}

// One verify pass (Section 3.3): layers k+1..L over the B * k_spec kept rows, then the head.
static dvi_status verify_pass(dvi_ctx *x, int nck, bool direct = false) {
    const dvi_config &cf = x->cfg;
    const int B = x->B, k = x->k_spec, M = B * k, d = cf.d_model;
    auto body = [&]() -> dvi_status {
        dvi_status sl =
            run_layers(x, cf.split_k, cf.n_layers, B, k, 0, nck, x->hk, x->hk_ss, x->hk_hg, 1, x->hk_hg, 1, 0);
        if (sl != DVI_OK) return sl;
        head(x, x->hk_hg, x->hk_ss, d / 16, M, x->vlogits, false, x->targets, 1, nullptr);
        LAUNCHCHK(x);
        return DVI_OK;
    };
    const dvi_status st = direct ? body() : run_pass(x, {1, B, k, 0, nck}, body);
    if (st != DVI_OK) return st;
    LAUNCHCHK(x);
    return DVI_OK;
}

// The commit kernel and the ring copy of the rows it logs.  limit: x->max_new holds each
// sequence's remaining tokens; dec: the kernel subtracts what it commits (several steps in a row).
static dvi_status commit_launch(dvi_ctx *x, bool limit, bool dec, int32_t *tok, int32_t *n, int32_t *m) {
    const dvi_config &cf = x->cfg;
    const int B = x->B, k = x->k_spec;
    CommitArgs a{};
    a.B = B;
    a.k_spec = k;
    a.drafts = x->drafts;
    a.targets = x->targets;
    a.max_new = limit ? x->max_new : nullptr;
    a.max_new_dec = dec ? 1 : 0;
    a.lens = x->lens;
    a.pending = x->pending;
    a.tokens_out = tok;
    a.n_out = n;
    a.m_out = m;
    a.flags = flags_ptr(x);
    a.ring_state = x->ring_state;
    a.ring_rows = x->ar_mode ? 0 : cf.buffer_rows;
    a.copy_list = x->copy_list;
    a.ring_a = x->ring_a;
    a.ring_i = x->ring_i;
    a.ring_prev = x->ring_prev;
    a.ring_r = x->ring_r;
    a.ring_fresh = x->ring_fresh;
    a.rng_step = x->rng_step;
    if (x->ar_mode) {
        // plain autoregressive step: nothing was drafted; commit y*_1 only
        HIPCHK(x, hipMemsetAsync(x->drafts, 0xff, (size_t)B * 4, x->stream));
    }
    launch_commit(a, x->stream);
    if (!x->ar_mode)
        launch_ring_copy(x->copy_list, B * k, x->hk_hat, cf.d_model, (int)x->es, x->vlogits, cf.vocab, x->ring_h,
                         x->ring_logits, x->stream);
    LAUNCHCHK(x);
    return DVI_OK;
}

extern "C" dvi_status dvi_draft(dvi_ctx *x, int32_t k_spec, const int32_t *forced, int32_t *drafts_out) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_READY) return fail(x, DVI_ERR_STATE, "draft needs state READY");
    const dvi_config &cf = x->cfg;
    if (k_spec < 1) return fail(x, DVI_ERR_ARG, "k_spec < 1");
    if (k_spec > cf.max_k_spec) return fail(x, DVI_ERR_CAPACITY, "k_spec %d > max_k_spec %d", k_spec, cf.max_k_spec);
    for (int b = 0; b < x->B; ++b)
        if (x->lens_h[b] + k_spec > cf.max_seq)
            return fail(x, DVI_ERR_CAPACITY, "sequence %d: length %d + k_spec %d > max_seq %d", b, x->lens_h[b], k_spec,
                        cf.max_seq);
    const int B = x->B;
    if (forced) {
        for (int i = 0; i < B * k_spec; ++i)
            if (forced[i] < 0 || forced[i] >= cf.vocab) return fail(x, DVI_ERR_ARG, "forced draft id out of range");
        HIPCHK(x, hipMemcpyAsync(x->forced, forced, (size_t)B * k_spec * 4, hipMemcpyHostToDevice, x->stream));
    }
    ev_begin(x, 0);
    HIPCHK(x, hipMemsetAsync(flags_ptr(x), 0, 16, x->stream));
    const dvi_status st = draft_pass(x, k_spec, forced != nullptr, attn_chunks(x, max_len(x) + k_spec - 1));
    if (st != DVI_OK) return st;
    ev_end(x, 0);
    if (drafts_out) {
        HIPCHK(x, hipMemcpyAsync(drafts_out, x->drafts, (size_t)B * k_spec * 4, hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipStreamSynchronize(x->stream));
    }
    x->state = S_DRAFTED;
    return DVI_OK;
}

extern "C" dvi_status dvi_verify(dvi_ctx *x, int32_t *targets_out, int32_t *accept_out) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_DRAFTED) return fail(x, DVI_ERR_STATE, "verify needs state DRAFTED");
    const int B = x->B, k = x->k_spec, M = B * k;
    ev_begin(x, 1);
    const dvi_status st = verify_pass(x, attn_chunks(x, max_len(x) + k - 1));
    if (st != DVI_OK) return st;
    ev_end(x, 1);
    if (targets_out || accept_out) {
        std::vector<int32_t> tg((size_t)M), dr((size_t)M);
        HIPCHK(x, hipMemcpyAsync(tg.data(), x->targets, (size_t)M * 4, hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipMemcpyAsync(dr.data(), x->drafts, (size_t)(x->ar_mode ? B : M) * 4, hipMemcpyDeviceToHost,
                                 x->stream));
        HIPCHK(x, hipStreamSynchronize(x->stream));
        if (targets_out) memcpy(targets_out, tg.data(), (size_t)M * 4);
        if (accept_out)
            for (int b = 0; b < B; ++b) {
                int m = 0;
                if (!x->ar_mode)
                    while (m < k && dr[(size_t)b * k + m] == tg[(size_t)b * k + m]) ++m;
                accept_out[b] = m;
            }
    }
    x->state = S_VERIFIED;
    return DVI_OK;
}

// Bytes of static scratch one verify of M rows over nck attention chunks takes (each piece
// 256-byte aligned), and its layout when base is given.
static size_t static_scratch_layout(const dvi_ctx *x, int M, int nck, void *base, Scratch *out) {
    const dvi_config &c = x->cfg;
    Bump b(base);
    Scratch s;
    s.chunk_stride = nck;
    s.att_po = b.take<float>((size_t)M * c.n_heads * nck * c.head_dim * 4);
    s.att_pml = b.take<float>((size_t)M * c.n_heads * nck * 2 * 4);
    s.att_cnt = b.take<int32_t>((size_t)c.max_batch * c.n_kv_heads * kCounterStride * 4);
    s.part_val = b.take<float>((size_t)M * (c.vocab / 16) * 4);
    s.part_idx = b.take<int32_t>((size_t)M * (c.vocab / 16) * 4);
    if (out) *out = s;
    return align_up(b.off);
}

extern "C" dvi_status dvi_verify_static(dvi_ctx *x, int32_t *targets_out, int32_t *accept_out) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_DRAFTED) return fail(x, DVI_ERR_STATE, "verify needs state DRAFTED");
    if (!x->static_scratch) return fail(x, DVI_ERR_DEVICE, "the static scratch of device %d is not available", x->dev);
    const int B = x->B, k = x->k_spec, M = B * k;
    const int nck = attn_chunks(x, max_len(x) + k - 1);
    const size_t need = static_scratch_layout(x, M, nck, nullptr, nullptr);
    if (need > kStaticScratchBytes)
        return fail(x, DVI_ERR_CAPACITY, "verify of %d rows over %d key chunks needs %zu bytes of static scratch; the maximum is %zu",
                    M, nck, need, kStaticScratchBytes);
    Scratch st_scr;
    static_scratch_layout(x, M, nck, x->static_scratch, &st_scr);
    // the merge counters start at zero (a kernel, not a memset, so a caller may capture this call)
    const int ncnt = x->cfg.max_batch * x->cfg.n_kv_heads * kCounterStride;
    fill_i32_kernel<<<(ncnt + 255) / 256, 256, 0, x->stream>>>(st_scr.att_cnt, ncnt, 0);
    LAUNCHCHK(x);
    ev_begin(x, 1);
    x->scr = st_scr;
    const dvi_status st = verify_pass(x, nck, true);
    x->scr = x->ws_scr;
    if (st != DVI_OK) return st;
    ev_end(x, 1);
    if (targets_out || accept_out) {
        int32_t tg[kMaxRows], dr[kMaxRows];  // M <= kMaxRows (max_batch * max_k_spec is checked at create)
        HIPCHK(x, hipMemcpyAsync(tg, x->targets, (size_t)M * 4, hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipMemcpyAsync(dr, x->drafts, (size_t)(x->ar_mode ? B : M) * 4, hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipStreamSynchronize(x->stream));
        if (targets_out) memcpy(targets_out, tg, (size_t)M * 4);
        if (accept_out)
            for (int b = 0; b < B; ++b) {
                int m = 0;
                if (!x->ar_mode)
                    while (m < k && dr[b * k + m] == tg[b * k + m]) ++m;
                accept_out[b] = m;
            }
    }
    x->state = S_VERIFIED;
    return DVI_OK;
}

extern "C" dvi_status dvi_commit(dvi_ctx *x, const int32_t *max_new, const int32_t *forced_commit, int32_t *tokens_out,
                                 int32_t *n_out, int32_t *accept_out) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_VERIFIED) return fail(x, DVI_ERR_STATE, "commit needs state VERIFIED");
    if (!tokens_out || !n_out) return fail(x, DVI_ERR_ARG, "null output");
    const dvi_config &cf = x->cfg;
    const int B = x->B, k = x->k_spec;
    if (forced_commit) {
        for (int i = 0; i < B * k; ++i)
            if (forced_commit[i] < 0 || forced_commit[i] >= cf.vocab)
                return fail(x, DVI_ERR_ARG, "forced commit id out of range");
        HIPCHK(x, hipMemcpyAsync(x->targets, forced_commit, (size_t)B * k * 4, hipMemcpyHostToDevice, x->stream));
    }
    if (max_new) {
        for (int b = 0; b < B; ++b)
            if (max_new[b] < 0) return fail(x, DVI_ERR_ARG, "max_new < 0");
        HIPCHK(x, hipMemcpyAsync(x->max_new, max_new, (size_t)B * 4, hipMemcpyHostToDevice, x->stream));
    }
    ev_begin(x, 2);
    const dvi_status st = commit_launch(x, max_new != nullptr, false, x->io, x->io + io_n(x), x->io + io_m(x));
    if (st != DVI_OK) return st;
    ev_end(x, 2);
    std::vector<int32_t> io((size_t)io_words(x));
    HIPCHK(x, hipMemcpyAsync(io.data(), x->io, io.size() * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    // Non-finite logits: the commit kernel committed nothing; the caller aborts the step.
    if (io[io_flags(x)]) return fail(x, DVI_ERR_NUMERIC, "non-finite logits in the draft or verify head");
    memcpy(tokens_out, io.data(), (size_t)B * k * 4);
    memcpy(n_out, io.data() + io_n(x), (size_t)B * 4);
    if (accept_out) memcpy(accept_out, io.data() + io_m(x), (size_t)B * 4);
    for (int b = 0; b < B; ++b) {
        x->lens_h[b] += io[io_n(x) + b];
        const int m = io[io_m(x) + b];
        const bool logged = !x->ar_mode && (!max_new || max_new[b] > 0);
        if (logged) {
            x->ring_valid_h += (m + 1 < k ? m + 1 : k);
            if (x->ring_valid_h > cf.buffer_rows) x->ring_valid_h = cf.buffer_rows;
        }
    }
    x->state = S_READY;
    return DVI_OK;
}

extern "C" dvi_status dvi_decode_steps(dvi_ctx *x, int32_t k_spec, int32_t n_steps, const int32_t *max_new,
                                       int32_t *tokens_out, int32_t *n_out, int32_t *accept_out) {
    if (!x) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_READY) return fail(x, DVI_ERR_STATE, "decode_steps needs state READY");
    if (!tokens_out || !n_out) return fail(x, DVI_ERR_ARG, "null output");
    const dvi_config &cf = x->cfg;
    const int B = x->B;
    if (k_spec < 1) return fail(x, DVI_ERR_ARG, "k_spec < 1");
    if (k_spec > cf.max_k_spec) return fail(x, DVI_ERR_CAPACITY, "k_spec %d > max_k_spec %d", k_spec, cf.max_k_spec);
    if (n_steps < 1 || n_steps > kMaxDecodeSteps)
        return fail(x, DVI_ERR_ARG, "n_steps %d outside 1..%d", n_steps, kMaxDecodeSteps);
    if (max_new)
        for (int b = 0; b < B; ++b)
            if (max_new[b] < 0) return fail(x, DVI_ERR_ARG, "max_new < 0");
    // A sequence grows by at most k_spec per step and by at most its max_new in all; each step's
    // drafts write k_spec positions past the length it starts from.
    auto grown = [&](int b, int steps) {
        const long g = (long)steps * k_spec;
        return (int)(max_new && max_new[b] < g ? max_new[b] : g);
    };
    for (int b = 0; b < B; ++b)
        if (x->lens_h[b] + grown(b, n_steps - 1) + k_spec > cf.max_seq)
            return fail(x, DVI_ERR_CAPACITY, "sequence %d: length %d may reach %d after %d steps of %d > max_seq %d", b,
                        x->lens_h[b], x->lens_h[b] + grown(b, n_steps - 1) + k_spec, n_steps, k_spec, cf.max_seq);
    if (max_new) HIPCHK(x, hipMemcpyAsync(x->max_new, max_new, (size_t)B * 4, hipMemcpyHostToDevice, x->stream));
    HIPCHK(x, hipMemsetAsync(flags_ptr(x), 0, 16, x->stream));
    const int Bk = B * k_spec;
    int32_t *tok_d = x->steps_io, *n_d = tok_d + (size_t)n_steps * Bk, *m_d = n_d + (size_t)n_steps * B;
    for (int st = 0; st < n_steps; ++st) {
        // the attention grid covers the longest length this step can start from
        int pmax = 0;
        for (int b = 0; b < B; ++b) pmax = std::max(pmax, x->lens_h[b] + grown(b, st));
        const int nck = attn_chunks(x, pmax + k_spec - 1);
        dvi_status s = draft_pass(x, k_spec, false, nck);
        if (s == DVI_OK) s = verify_pass(x, nck);
        if (s == DVI_OK)
            s = commit_launch(x, max_new != nullptr, true, tok_d + (size_t)st * Bk, n_d + (size_t)st * B,
                              m_d + (size_t)st * B);
        if (s != DVI_OK) return s;
    }
    std::vector<int32_t> io((size_t)n_steps * (Bk + 2 * B)), fl(4), rs(4);
    HIPCHK(x, hipMemcpyAsync(io.data(), x->steps_io, io.size() * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipMemcpyAsync(fl.data(), flags_ptr(x), 16, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipMemcpyAsync(rs.data(), x->ring_state, 16, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    const int32_t *tok = io.data(), *nn = tok + (size_t)n_steps * Bk, *mm = nn + (size_t)n_steps * B;
    memcpy(tokens_out, tok, (size_t)n_steps * Bk * 4);
    memcpy(n_out, nn, (size_t)n_steps * B * 4);
    if (accept_out) memcpy(accept_out, mm, (size_t)n_steps * B * 4);
    // host mirrors of the lengths and of the ring's valid rows
    for (int st = 0; st < n_steps; ++st)
        for (int b = 0; b < B; ++b) x->lens_h[b] += nn[(size_t)st * B + b];
    x->ring_valid_h = rs[1];
    x->state = S_READY;
    // Non-finite logits: the commit kernel commits nothing from that step on; the earlier steps
    // stand, and the context stays usable from the lengths they reached.
    if (fl[0]) return fail(x, DVI_ERR_NUMERIC, "non-finite logits in the draft or verify head");
    return DVI_OK;
}

extern "C" dvi_status dvi_abort_step(dvi_ctx *x) {
    if (!x) return DVI_ERR_ARG;
    if (x->state != S_DRAFTED && x->state != S_VERIFIED) return fail(x, DVI_ERR_STATE, "no step in progress");
    HIPCHK(x, hipMemsetAsync(flags_ptr(x), 0, 16, x->stream));
    x->state = S_READY;
    return DVI_OK;
}

// ------------------------------------------------------------------------------------------
// C ABI: drafter update
// ------------------------------------------------------------------------------------------
__global__ void clear_i8_kernel(int8_t *p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

extern "C" dvi_status dvi_update_drafter(dvi_ctx *x, const dvi_update_args *ua, dvi_update_stats *stats) {
    if (!x || !ua) return DVI_ERR_ARG;
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    if (x->state != S_READY) return fail(x, DVI_ERR_STATE, "update needs state READY");
    if (!(ua->tau > 0.f)) return fail(x, DVI_ERR_ARG, "tau must be > 0");
    if (ua->lr != 0.f && ua->opt_step < 1) return fail(x, DVI_ERR_ARG, "opt_step must be >= 1");
    const dvi_config &cf = x->cfg;
    const int n = x->ring_valid_h;
    if (stats) memset(stats, 0, sizeof(*stats));
    if (n == 0) return DVI_OK;
    ev_begin(x, 3);
    UpdateArgs u{};
    u.W = x->head;
    u.Hh = x->ring_h;
    u.logits = x->ring_logits;
    u.a = x->ring_a;
    u.r = x->ring_r;
    u.fresh = x->ring_fresh;
    u.n = n;
    u.V = cf.vocab;
    u.d = cf.d_model;
    u.rank = cf.lora_rank;
    u.gamma = cf.lora_gamma;
    u.tau = ua->tau;
    u.baseline = ua->baseline;
    u.c_kl = ua->c_kl;
    u.c_ce = ua->c_ce;
    u.c_pg = ua->c_pg;
    u.c_ent = ua->c_ent;
    u.A = x->lora_A;
    u.Bm = x->lora_B;
    u.u = x->upd_u;
    u.Z = x->upd_Z;
    u.part_val = x->ws_scr.part_val;
    u.part_idx = x->ws_scr.part_idx;
    u.row_stats = x->upd_stats;
    u.dA = x->upd_dA;
    u.du = x->upd_du;
    u.du_part = x->upd_dup;
    u.dB = x->upd_dB;
    u.loss_out = x->upd_loss;
    u.xfm = x->ufm;
    launch_update_forward(x->dt, u, x->stream);
    launch_update_backward(x->dt, u, x->stream);
    const size_t nA = (size_t)cf.vocab * cf.lora_rank, nB = (size_t)cf.lora_rank * cf.d_model;
    if (ua->grad_A_out)
        HIPCHK(x, hipMemcpyAsync(ua->grad_A_out, x->upd_dA, nA * 4, hipMemcpyDeviceToDevice, x->stream));
    if (ua->grad_B_out)
        HIPCHK(x, hipMemcpyAsync(ua->grad_B_out, x->upd_dB, nB * 4, hipMemcpyDeviceToDevice, x->stream));
    if (ua->lr != 0.f) {
        launch_adam(x->lora_A, x->upd_dA, x->mA, x->vA, (int)nA, ua->lr, ua->beta1, ua->beta2, ua->eps, ua->opt_step,
                    x->stream);
        launch_adam(x->lora_B, x->upd_dB, x->mB, x->vB, (int)nB, ua->lr, ua->beta1, ua->beta2, ua->eps, ua->opt_step,
                    x->stream);
    }
    clear_i8_kernel<<<(cf.buffer_rows + 255) / 256, 256, 0, x->stream>>>(x->ring_fresh, cf.buffer_rows);
    ev_end(x, 3);
    LAUNCHCHK(x);
    float lo[16];
    HIPCHK(x, hipMemcpyAsync(lo, x->upd_loss, 16 * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    if (stats) {
        stats->loss = lo[0];
        stats->kl = lo[1];
        stats->ce = lo[2];
        stats->pg = lo[3];
        stats->entropy = lo[4];
        stats->rows = (int32_t)lo[5];
        stats->accepted = (int32_t)lo[6];
        stats->fresh = (int32_t)lo[7];
        stats->fresh_accepted = (int32_t)lo[8];
    }
    return DVI_OK;
}

// ------------------------------------------------------------------------------------------
// C ABI: inspection and test hooks
// ------------------------------------------------------------------------------------------
extern "C" dvi_status dvi_read_kv(dvi_ctx *x, int32_t layer, int32_t seq, int32_t pos0, int32_t npos, void *k, void *v) {
    if (!x || !k || !v) return DVI_ERR_ARG;
    const dvi_config &cf = x->cfg;
    if (layer < 0 || layer >= cf.n_layers || seq < 0 || seq >= cf.max_batch || pos0 < 0 || npos < 0 ||
        pos0 + npos > cf.max_seq)
        return fail(x, DVI_ERR_ARG, "read_kv range");
    const size_t es = x->es, hd = cf.head_dim, cap = x->s_cap;
    if (npos == 0) return DVI_OK;
    // both caches are stored in fragment-major blocks of 64 positions: fetch the whole blocks
    // that cover the range, then gather [n_kv][npos][hd]
    const int c0 = pos0 / 64, nc = (pos0 + npos - 1) / 64 - c0 + 1, kc = pack_kc(x->dt);
    const size_t cbytes = hd * 64 * es;
    std::vector<uint8_t> kt((size_t)cf.n_kv_heads * nc * cbytes), vt(kt.size());
    for (int h = 0; h < cf.n_kv_heads; ++h) {
        const size_t off = (((size_t)seq * cf.n_kv_heads + h) * cap + (size_t)c0 * 64) * hd * es;
        HIPCHK(x, hipMemcpyAsync(kt.data() + (size_t)h * nc * cbytes, (uint8_t *)x->L[layer].Kc + off, nc * cbytes,
                                 hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipMemcpyAsync(vt.data() + (size_t)h * nc * cbytes, (uint8_t *)x->L[layer].Vc + off, nc * cbytes,
                                 hipMemcpyDeviceToHost, x->stream));
    }
    HIPCHK(x, hipStreamSynchronize(x->stream));
    for (int h = 0; h < cf.n_kv_heads; ++h)
        for (int p = 0; p < npos; ++p) {
            const int pa = pos0 + p, c = pa / 64 - c0, o = pa % 64;
            const size_t blk = ((size_t)h * nc + c) * cbytes, dst = ((size_t)h * npos + p) * hd * es;
            for (int d = 0; d < (int)hd; ++d) {
                memcpy((uint8_t *)k + dst + d * es, kt.data() + blk + kv_key_offset(kc, (int)hd, o, d) * es, es);
                memcpy((uint8_t *)v + dst + d * es, vt.data() + blk + kv_val_offset(kc, (int)hd, o, d) * es, es);
            }
        }
    return DVI_OK;
}

extern "C" dvi_status dvi_read_logits(dvi_ctx *x, float *out) {
    if (!x || !out) return DVI_ERR_ARG;
    if (x->state != S_VERIFIED && x->state != S_READY) return fail(x, DVI_ERR_STATE, "no verify logits");
    HIPCHK(x, hipMemcpyAsync(out, x->vlogits, (size_t)x->B * x->k_spec * x->cfg.vocab * 4, hipMemcpyDeviceToHost,
                             x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    return DVI_OK;
}

extern "C" dvi_status dvi_read_draft_logits(dvi_ctx *x, float *out) {
    if (!x || !out) return DVI_ERR_ARG;
    HIPCHK(x, hipMemcpyAsync(out, x->dlogits, (size_t)x->B * x->cfg.vocab * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    return DVI_OK;
}

extern "C" dvi_status dvi_read_lengths(dvi_ctx *x, int32_t *len) {
    if (!x || !len) return DVI_ERR_ARG;
    HIPCHK(x, hipMemcpyAsync(len, x->lens, (size_t)x->B * 4, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    return DVI_OK;
}

extern "C" dvi_status dvi_buffer_info(dvi_ctx *x, int32_t *valid, int32_t *next) {
    if (!x) return DVI_ERR_ARG;
    int32_t rs[4];
    HIPCHK(x, hipMemcpyAsync(rs, x->ring_state, 16, hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    if (valid) *valid = rs[1];
    if (next) *next = rs[0];
    return DVI_OK;
}

extern "C" dvi_status dvi_read_buffer(dvi_ctx *x, int32_t row0, int32_t nrows, float *h, int32_t *a, float *logits,
                                      int8_t *r, int8_t *fresh, int32_t *i, int32_t *prev) {
    if (!x) return DVI_ERR_ARG;
    const dvi_config &cf = x->cfg;
    if (row0 < 0 || nrows < 0 || row0 + nrows > cf.buffer_rows) return fail(x, DVI_ERR_ARG, "buffer range");
    const size_t d = cf.d_model, V = cf.vocab;
    if (h) {
        std::vector<uint8_t> tmp((size_t)nrows * d * x->es);
        HIPCHK(x, hipMemcpyAsync(tmp.data(), (uint8_t *)x->ring_h + (size_t)row0 * d * x->es, tmp.size(),
                                 hipMemcpyDeviceToHost, x->stream));
        HIPCHK(x, hipStreamSynchronize(x->stream));
        for (size_t e = 0; e < (size_t)nrows * d; ++e) {
            if (x->dt == DType::BF16) {
                uint32_t u = (uint32_t)((uint16_t *)tmp.data())[e] << 16;
                memcpy(&h[e], &u, 4);
            } else {
                h[e] = ((float *)tmp.data())[e];
            }
        }
    }
    if (a) HIPCHK(x, hipMemcpyAsync(a, x->ring_a + row0, nrows * 4, hipMemcpyDeviceToHost, x->stream));
    if (i) HIPCHK(x, hipMemcpyAsync(i, x->ring_i + row0, nrows * 4, hipMemcpyDeviceToHost, x->stream));
    if (prev) HIPCHK(x, hipMemcpyAsync(prev, x->ring_prev + row0, nrows * 4, hipMemcpyDeviceToHost, x->stream));
    if (r) HIPCHK(x, hipMemcpyAsync(r, x->ring_r + row0, nrows, hipMemcpyDeviceToHost, x->stream));
    if (fresh) HIPCHK(x, hipMemcpyAsync(fresh, x->ring_fresh + row0, nrows, hipMemcpyDeviceToHost, x->stream));
    if (logits)
        HIPCHK(x, hipMemcpyAsync(logits, x->ring_logits + (size_t)row0 * V, (size_t)nrows * V * 4,
                                 hipMemcpyDeviceToHost, x->stream));
    HIPCHK(x, hipStreamSynchronize(x->stream));
    return DVI_OK;
}

extern "C" dvi_status dvi_write_buffer(dvi_ctx *x, int32_t nrows, const float *h, const int32_t *a,
                                       const float *logits, const int8_t *r, const int8_t *fresh) {
    if (!x || !h || !a || !logits || !r || !fresh) return DVI_ERR_ARG;
    if (x->state == S_DRAFTED || x->state == S_VERIFIED) return fail(x, DVI_ERR_STATE, "write_buffer during a step");
    const dvi_config &cf = x->cfg;
    if (nrows < 1 || nrows > cf.buffer_rows) return fail(x, DVI_ERR_CAPACITY, "nrows out of range");
    const size_t d = cf.d_model, V = cf.vocab;
    for (int e = 0; e < nrows; ++e)
        if (a[e] < 0 || a[e] >= cf.vocab) return fail(x, DVI_ERR_ARG, "action id out of range");
    std::vector<uint8_t> tmp((size_t)nrows * d * x->es);
    for (size_t e = 0; e < (size_t)nrows * d; ++e) {
        if (x->dt == DType::BF16) {
            uint32_t u;
            memcpy(&u, &h[e], 4);
            if ((u & 0x7fffffffu) > 0x7f800000u) u = (u >> 16) | 0x40;
            else u = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
            ((uint16_t *)tmp.data())[e] = (uint16_t)u;
        } else {
            ((float *)tmp.data())[e] = h[e];
        }
    }
    std::vector<int32_t> zi(nrows, 0), neg(nrows, -1);
    HIPCHK(x, hipMemcpy(x->ring_h, tmp.data(), tmp.size(), hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_logits, logits, (size_t)nrows * V * 4, hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_a, a, nrows * 4, hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_i, zi.data(), nrows * 4, hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_prev, neg.data(), nrows * 4, hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_r, r, nrows, hipMemcpyHostToDevice));
    HIPCHK(x, hipMemcpy(x->ring_fresh, fresh, nrows, hipMemcpyHostToDevice));
    int32_t rs[4] = {nrows % cf.buffer_rows, nrows, 0, 0};
    HIPCHK(x, hipMemcpy(x->ring_state, rs, 16, hipMemcpyHostToDevice));
    x->ring_valid_h = nrows;
    return DVI_OK;
}

extern "C" dvi_status dvi_probe_kernel(dvi_ctx *x, int32_t which) {
    if (!x) return DVI_ERR_ARG;
    if (which < DVI_PROBE_OFF || which > DVI_PROBE_ATTENTION) return fail(x, DVI_ERR_ARG, "unknown probe %d", which);
    if (which != DVI_PROBE_OFF && x->pev.empty()) {
        x->pev.resize(2 * kProbeMax);
        for (auto &e : x->pev) HIPCHK(x, hipEventCreate(&e));
    }
    HIPCHK(x, hipStreamSynchronize(x->stream));
    x->probe = which;
    x->pused = 0;
    x->plaunch = 0;
    x->pbytes = 0.0;
    return DVI_OK;
}

extern "C" dvi_status dvi_probe_read(dvi_ctx *x, double *total_ms, int64_t *launches, double *bytes) {
    if (!x) return DVI_ERR_ARG;
    HIPCHK(x, hipStreamSynchronize(x->stream));
    double t = 0.0;
    for (size_t i = 0; i + 1 < x->pused; i += 2) {
        float ms = 0.f;
        HIPCHK(x, hipEventElapsedTime(&ms, x->pev[i], x->pev[i + 1]));
        t += ms;
    }
    if (total_ms) *total_ms = t;
    if (launches) *launches = x->plaunch;
    if (bytes) *bytes = x->pbytes;
    return DVI_OK;
}

extern "C" dvi_status dvi_measure_read_rate(dvi_ctx *x, const void *buf, size_t bytes, int32_t reps, double *gb_s) {
    if (!x) return DVI_ERR_ARG;
    if (!buf || !gb_s || reps < 1 || bytes < ((size_t)1 << 20) || bytes % 16)
        return fail(x, DVI_ERR_ARG, "read-rate buffer must be >= 1 MiB and a multiple of 16 bytes, reps >= 1");
    if (x->device_error) return fail(x, DVI_ERR_DEVICE, "context has a sticky device error");
    hipEvent_t e0, e1;
    HIPCHK(x, hipEventCreate(&e0));
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return fail(x, DVI_ERR_DEVICE, "hipEventCreate failed");
    }
    double best = 0.0;
    dvi_status st = DVI_OK;
    for (int r = 0; r < reps && st == DVI_OK; ++r) {
        LaunchEvents ev;
        ev.start = e0;
        ev.stop = e1;
        launch_stream_read(buf, bytes, (uint32_t *)(x->rng_step + 2), x->stream, ev);
        float ms = 0.f;
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&ms, e0, e1) != hipSuccess)
            st = fail(x, DVI_ERR_DEVICE, "read-rate pass failed");
        else if (ms > 0.f)
            best = std::max(best, (double)bytes / (ms * 1e-3) / 1e9);
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (st == DVI_OK) *gb_s = best;
    return st;
}

extern "C" dvi_status dvi_get_timings(dvi_ctx *x, double *md, double *mv, double *mc, double *mu) {
    if (!x) return DVI_ERR_ARG;
    double *outs[4] = {md, mv, mc, mu};
    for (int p = 0; p < 4; ++p) {
        if (x->ev_ok && x->ev_pending[p]) {
            float ms = 0.f;
            HIPCHK(x, hipEventSynchronize(x->ev[2 * p + 1]));
            HIPCHK(x, hipEventElapsedTime(&ms, x->ev[2 * p], x->ev[2 * p + 1]));
            x->ms[p] = ms;
            x->ev_pending[p] = 0;
        }
        if (outs[p]) *outs[p] = x->ms[p];
    }
    return DVI_OK;
}
