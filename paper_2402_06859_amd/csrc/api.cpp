// Host side of the librdcn C ABI (declared in include/rdcn.h): argument
// validation, workspace layouts, and the order of kernel launches for the
// gather, the Residual-DCN forward and backward, and the embedding backward.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <new>
#include <string.h>
#include <vector>

#include "../../include/rdcn.h"
#include "embed_bwd.h"
#include "gemm.h"
#include "head.h"
#include "kernels.h"

struct rdcn_handle {
    rdcn_config cfg;
    int64_t d;
    int n;   // projections per layer (3 with the attention term, 4 with parallel branches, else 1)
    int hr;  // width of the up projection's input (2r with parallel branches, else r)
    bool bf16, ids64, attn, par;
    bool split;  // activation mode 1: x_l (l >= 1) and h as bf16 hi + lo pairs
    bool f16;    // activation mode 2: x_l (l >= 1) and h as f16 (plus bf16 copies for the weight gradients)
    bool side_enabled = true;  // rdcn_set_side_stream
    uint32_t magic, shift;
    // the backward's weight-gradient products run on `side`, forked from and joined
    // back to the caller's stream with these events (no timing)
    hipStream_t side = nullptr;
    hipEvent_t ev_pw = nullptr, ev_att = nullptr, ev_side[2] = {nullptr, nullptr}, ev_join = nullptr;
    int* err;  // device error word
    void* static_scratch = nullptr;  // this device's qr_embed_backward_static workspace
    bool head_on = false;
    rdcn_head_config head{};
    // per-kernel timing (rdcn_profile_start / rdcn_profile_stop)
    bool prof_on = false;
    uint32_t prof_mask = 0;
    std::vector<hipEvent_t> prof_ev;   // 2 per launch
    std::vector<int> prof_kind;        // kernel of each recorded pair
    size_t prof_used = 0;
};

namespace {

// Brackets the launches of one kernel with an event pair when timing is on.
struct ProfScope {
    rdcn_handle* h;
    hipStream_t s;
    bool active;
    ProfScope(rdcn_handle* hh, int kind, hipStream_t ss) : h(hh), s(ss), active(false) {
        if (h->prof_on && ((h->prof_mask >> kind) & 1u) && 2 * (h->prof_used + 1) <= h->prof_ev.size()) {
            active = hipEventRecord(h->prof_ev[2 * h->prof_used], s) == hipSuccess;
            if (active) h->prof_kind.push_back(kind);
        }
    }
    ~ProfScope() {
        if (active) {
            (void)hipEventRecord(h->prof_ev[2 * h->prof_used + 1], s);
            ++h->prof_used;
        }
    }
};

}  // namespace

namespace {

using namespace rdcn;

constexpr size_t ALIGN = 256;
inline size_t al(size_t x) { return (x + ALIGN - 1) & ~(ALIGN - 1); }

inline rdcn_status hip_status(hipError_t e) { return e == hipSuccess ? RDCN_OK : RDCN_ERR_HIP; }
#define RDCN_TRY(expr)                                   \
    do {                                                 \
        hipError_t _e = (expr);                          \
        if (_e != hipSuccess) return RDCN_ERR_HIP;       \
    } while (0)

// Granlund-Montgomery magic number for unsigned 32-bit division by m >= 1.
void div_magic_host(uint32_t m, uint32_t& magic, uint32_t& shift) {
    if (m <= 1) {
        magic = 1;
        shift = 0;
        return;
    }
    uint32_t l = 0;
    while (((uint64_t)1 << l) < m) ++l;  // l = ceil(log2 m)
    magic = (uint32_t)((((uint64_t)1 << 32) * (((uint64_t)1 << l) - m)) / m + 1);
    shift = l - 1;
}

size_t eb(const rdcn_handle* h) { return h->bf16 ? 2 : 4; }

// Per layer: [v|q|k] (float with the attention term, else storage; plus a second
// plane of v without it), h and its second plane (attention only), the attention row
// statistics [o | Z | W1 | W2] (float, bf16 storage with attention), t, x_{l+1} and its
// second plane (l < L-1). Second planes exist with activation modes 1 (the lo part of a
// bf16 hi + lo pair) and 2: x_{l+1} is then f16 in X and its bf16 copy (the weight
// gradient's operand) in X2, h is bf16 in H and f16 in H2, and v (no attention) bf16 in
// P and f16 in P2.
struct SavedLayout {
    size_t P[RDCN_MAX_LAYERS], P2[RDCN_MAX_LAYERS], H[RDCN_MAX_LAYERS], H2[RDCN_MAX_LAYERS], A[RDCN_MAX_LAYERS],
        T[RDCN_MAX_LAYERS], X[RDCN_MAX_LAYERS], X2[RDCN_MAX_LAYERS];
    size_t total;
};

SavedLayout saved_layout(const rdcn_handle* h, int64_t B) {
    SavedLayout s;
    const size_t e = eb(h), d = (size_t)h->d, r = (size_t)h->cfg.rank, n = (size_t)h->n;
    const bool sp = h->split || h->f16;
    size_t off = 0;
    for (int l = 0; l < h->cfg.num_layers; ++l) {
        const bool more = l + 1 < h->cfg.num_layers;
        // float [v|q|k] feeds the attention (with parallel branches the plain branch's
        // value goes straight into the first half of H instead)
        s.P[l] = off; off += al(B * (h->par ? 3 : n) * r * (h->attn ? 4 : e));
        s.P2[l] = off; off += (sp && !h->attn) ? al(B * r * e) : 0;
        s.H[l] = off; off += h->attn ? al(B * (size_t)h->hr * e) : 0;
        s.H2[l] = off; off += (sp && h->attn) ? al(B * r * e) : 0;
        s.A[l] = off; off += (h->attn && h->bf16) ? al(B * 4 * r * 4) : 0;
        s.T[l] = off; off += al(B * d * e);
        s.X[l] = off; off += more ? al(B * d * e) : 0;  // x_{l+1}
        s.X2[l] = off; off += (sp && more) ? al(B * d * e) : 0;
    }
    s.total = off;
    return s;
}

// gt, gP and part alternate between two copies by layer parity: the side stream
// still reads layer l's copies while the main stream computes layer l - 1.
struct ScratchLayout {
    size_t g, gt[2], gh, gP[2], part[2], splitk, total;
    int nrb;
};

// Split-K target of the backward's weight-gradient GEMMs, which run on the side
// stream beside the main chain. Below 8e9 multiply-adds fewer splits leave more of
// the chip to the main stream and shrink the partials the reduction reads (384, the
// full-chip target: 0.749 ms per small step; 192: 0.733; 128: 0.726; 64: slower
// again); larger products (feed: 3.7e10) outlast the main chain with fewer splits
// (4.23 -> 4.81 ms per feed step at 128) and keep 384.
int bwd_split_blocks(int64_t M, int64_t N, int64_t K) {
    return (double)M * (double)N * (double)K < 8.0e9 ? 128 : 384;
}

int64_t splitk_elems(const rdcn_handle* h, int64_t B) {
    const int64_t d = h->d, r = h->cfg.rank, nr = (int64_t)h->n * r, hr = h->hr;
    const GemmPlan pu = plan_gemm(d, hr, B, h->bf16, true, bwd_split_blocks(d, hr, B));
    const GemmPlan pw = plan_gemm(nr, d, B, h->bf16, true, bwd_split_blocks(nr, d, B));
    int64_t m = 0;
    if (pu.splits > 1) m = pu.splits * d * hr;
    if (pw.splits > 1 && pw.splits * nr * d > m) m = pw.splits * nr * d;
    return m;
}

ScratchLayout scratch_layout(const rdcn_handle* h, int64_t B) {
    ScratchLayout s;
    const size_t e = eb(h), d = (size_t)h->d, r = (size_t)h->cfg.rank, n = (size_t)h->n;
    s.nrb = B > 0 ? (int)((B + pointwise_rows_per_block(B, d) - 1) / pointwise_rows_per_block(B, d)) : 0;
    const int copies = h->cfg.num_layers > 1 ? 2 : 1;
    size_t off = 0;
    s.g = off; off += al(B * d * 4);
    s.gh = off; off += h->attn ? al(B * r * 4) : 0;
    for (int k = 0; k < 2; ++k) {
        if (k >= copies) {
            s.gt[k] = s.gt[0];
            s.gP[k] = s.gP[0];
            s.part[k] = s.part[0];
            continue;
        }
        s.gt[k] = off; off += al(B * d * e);
        s.gP[k] = off; off += al(B * n * r * e);
        s.part[k] = off; off += al((size_t)s.nrb * d * 4);
    }
    s.splitk = off; off += al((size_t)splitk_elems(h, B) * 4);
    s.total = off;
    return s;
}

// Forward scratch (activation mode 2 only): one layer's weights converted to f16, the
// operands of the f16 projections (reused layer after layer).
struct FwdScratchLayout {
    size_t w16, u16, total;
};

FwdScratchLayout fwd_scratch_layout(const rdcn_handle* h) {
    FwdScratchLayout f{0, 0, 0};
    if (!h->f16) return f;
    const size_t d = (size_t)h->d;
    f.w16 = 0;
    f.u16 = al((size_t)h->n * h->cfg.rank * d * 2);
    f.total = f.u16 + al(d * (size_t)h->hr * 2);
    return f;
}

bool aligned256(const void* p) { return ((uintptr_t)p & 255u) == 0; }

rdcn_status check_batch(const rdcn_handle* h, int64_t batch) {
    if (!h) return RDCN_ERR_ARG;
    if (batch < 0) return RDCN_ERR_ARG;
    if (batch > h->cfg.batch_max) return RDCN_ERR_SHAPE;
    return RDCN_OK;
}

// One GEMM with split-K handled: writes the final float result to `out` (ldc = N).
hipError_t gemm_weight_grad(rdcn_handle* h, int kind, GemmArgs g, float* out, float* splitk, hipStream_t s,
                            int split_blocks = 384) {
    const GemmPlan p = plan_gemm(g.M, g.N, g.K, h->bf16, true, split_blocks);
    if (g.K == 0) return launch_fill_zero(out, g.M * g.N, s);
    g.ldc = g.N;
    if (p.splits == 1) {
        g.epi = EPI_STORE_F32;
        g.c = out;
        ProfScope ps(h, kind, s);
        return launch_gemm(g, p, h->bf16, s);
    }
    g.epi = EPI_PARTIAL;
    g.c = splitk;
    {
        ProfScope ps(h, kind, s);
        hipError_t e = launch_gemm(g, p, h->bf16, s);
        if (e != hipSuccess) return e;
    }
    ProfScope ps(h, RDCN_KERNEL_SPLITK_REDUCE, s);
    return launch_splitk_reduce(splitk, p.splits, g.M * g.N, out, s);
}

rdcn_status gather_args(rdcn_handle* h, int64_t batch, const void* ids, const int64_t* offsets,
                               const void* q_tables, const void* r_tables, const void* dense, void* x0,
                               GatherArgs& a) {
    const rdcn_config& c = h->cfg;
    if (!x0 || (c.num_cat > 0 && (!ids || !q_tables || !r_tables)) || (c.num_dense > 0 && !dense))
        return RDCN_ERR_ARG;
    a.batch = batch;
    a.F = c.num_cat;
    a.D = c.emb_dim;
    a.Nd = c.num_dense;
    a.rows_q = c.qr_rows_q;
    a.m = (uint32_t)c.qr_rows_r;
    a.vocab = (uint64_t)c.vocab;
    a.magic = h->magic;
    a.shift = h->shift;
    a.combine = c.combine == RDCN_COMBINE_MUL ? 0 : 1;
    a.hashed = c.hashed;
    a.seed = c.hash_seed;
    a.ids = ids;
    a.offsets = offsets;
    a.q_tables = q_tables;
    a.r_tables = r_tables;
    a.q_params = nullptr;
    a.r_params = nullptr;
    a.dense = dense;
    a.x0 = x0;
    a.err = h->err;
    return RDCN_OK;
}

// codes: 8 (bf16 models) or 4 (float) codes per lane load; params: float2 loads
bool q8_aligned(const rdcn_handle* h, const void* codes, const void* params) {
    const uintptr_t cm = h->bf16 ? 7u : 3u;
    return (((uintptr_t)codes) & cm) == 0 && (((uintptr_t)params) & 7u) == 0;
}

// ---------------------------------------------------------------------------
// Head layouts. Saved: per hidden layer a_l [B, n_l] twice, as bf16 (the weight
// gradients' operand and the ReLU masks) and as f16 (what the next layer, the gate
// logits and the logit read: three more mantissa bits keep the ReLU masks of the
// deeper layers close to those of the exact activations), (gated) s_l [B] float,
// then y [B] float and an f16 copy of the widest W_l (l >= 1) for the forward's
// f16 products. Scratch: two G planes [B, n_max] bf16 (the current layer's
// pre-activation gradient and the next one's), gy [B], two gs [B], the gate row
// partials, column-sum partials and split-K partials.
// ---------------------------------------------------------------------------
inline int64_t head_in(const rdcn_handle* h, int l) { return l == 0 ? h->d : h->head.hidden[l - 1]; }

struct HeadSaved {
    size_t A[RDCN_HEAD_MAX_HIDDEN], A16[RDCN_HEAD_MAX_HIDDEN], S[RDCN_HEAD_MAX_HIDDEN], Y, W16, total;
};

HeadSaved head_saved_layout(const rdcn_handle* h, int64_t B) {
    HeadSaved s;
    size_t off = 0, w16 = 0;
    for (int l = 0; l < h->head.num_hidden; ++l) {
        s.A[l] = off; off += al((size_t)B * h->head.hidden[l] * 2);
        s.A16[l] = off; off += al((size_t)B * h->head.hidden[l] * 2);
        s.S[l] = off; off += h->head.gated ? al((size_t)B * 4) : 0;
        if (l > 0) w16 = std::max(w16, (size_t)h->head.hidden[l] * h->head.hidden[l - 1] * 2);
    }
    s.Y = off; off += al((size_t)B * 4);
    s.W16 = off; off += al(w16);
    s.total = off;
    return s;
}

struct HeadScratch {
    size_t G[2], gy, gs, rowpart, colpart, splitk, total;  // gs: one [B] vector per layer
};

HeadScratch head_scratch_layout(const rdcn_handle* h, int64_t B) {
    const rdcn_head_config& c = h->head;
    int64_t nmax = 0, tiles = 0, split = 0, widest = std::max<int64_t>(h->d, c.num_buckets);
    for (int l = 0; l < c.num_hidden; ++l) {
        const int64_t nin = head_in(h, l), nout = c.hidden[l];
        nmax = std::max<int64_t>(nmax, nout);
        widest = std::max<int64_t>(widest, nout);
        if (l > 0) tiles = std::max<int64_t>(tiles, gemm_tiles_n(nin, plan_gemm(B, nin, nout, true, false)));
        const GemmPlan pw = plan_gemm(nout, nin, B, true, true);
        if (pw.splits > 1) split = std::max<int64_t>(split, pw.splits * nout * nin);
    }
    HeadScratch s;
    size_t off = 0;
    for (int i = 0; i < 2; ++i) { s.G[i] = off; off += al((size_t)B * nmax * 2); }
    s.gy = off; off += al((size_t)B * 4);
    s.gs = off; off += (size_t)c.num_hidden * al((size_t)B * 4);
    s.rowpart = off; off += c.gated ? al((size_t)tiles * B * 4) : 0;
    s.colpart = off; off += al((size_t)colsum_chunks(B) * widest * 4);
    s.splitk = off; off += al((size_t)split * 4);
    s.total = off;
    return s;
}

bool a16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

rdcn_status check_head_weights(const rdcn_handle* h, const rdcn_head_weights* w) {
    if (!w) return RDCN_ERR_ARG;
    const rdcn_head_config& c = h->head;
    for (int l = 0; l < c.num_hidden; ++l) {
        if (!w->w[l] || !w->b[l] || !a16(w->w[l]) || !a16(w->b[l])) return RDCN_ERR_ARG;
        if (c.gated && (!w->gate_w[l] || !w->gate_b[l] || !a16(w->gate_w[l]))) return RDCN_ERR_ARG;
    }
    if (!w->w_out || !w->b_out || !w->cal_w || !w->cal_b || !a16(w->w_out)) return RDCN_ERR_ARG;
    return RDCN_OK;
}

CalArgs cal_args(const rdcn_handle* h, const rdcn_head_weights* w, const float* e) {
    CalArgs c;
    c.K = h->head.num_buckets;
    c.lo = h->head.bucket_lo;
    c.step = h->head.bucket_step;
    c.w = (const float*)w->cal_w;
    c.b = (const float*)w->cal_b;
    c.e = e;
    return c;
}

}  // namespace

static_assert(RDCN_EMBED_STATIC_SCRATCH_BYTES == rdcn::EMB_STATIC_SCRATCH_BYTES,
              "the header states the static workspace size");

extern "C" {

const char* rdcn_status_string(rdcn_status s) {
    switch (s) {
        case RDCN_OK: return "ok";
        case RDCN_ERR_ARG: return "invalid argument";
        case RDCN_ERR_SHAPE: return "inconsistent shape";
        case RDCN_ERR_INDEX: return "id outside [0, vocab)";
        case RDCN_ERR_UNSUPPORTED: return "unsupported configuration";
        case RDCN_ERR_WORKSPACE: return "workspace too small or misaligned";
        case RDCN_ERR_HIP: return "HIP runtime error";
        case RDCN_ERR_RANGE: return "f16 activation beyond range";
    }
    return "unknown status";
}

rdcn_status rdcn_create(const rdcn_config* cfg, rdcn_handle** out) {
    if (!cfg || !out) return RDCN_ERR_ARG;
    *out = nullptr;
    const rdcn_config& c = *cfg;
    if (c.batch_max < 0 || c.num_cat < 0 || c.emb_dim <= 0 || c.num_dense < 0 || c.rank <= 0 ||
        c.num_layers < 1 || c.num_layers > RDCN_MAX_LAYERS || c.qr_rows_q <= 0 || c.qr_rows_r <= 0 ||
        (c.combine != RDCN_COMBINE_MUL && c.combine != RDCN_COMBINE_SUM) || (c.multi_hot != 0 && c.multi_hot != 1) ||
        (c.id_type != RDCN_I32 && c.id_type != RDCN_I64) || (c.dtype != RDCN_F32 && c.dtype != RDCN_BF16) ||
        (c.hashed != 0 && c.hashed != 1) || c.reserved2 != 0 || (c.hashed ? c.vocab != 0 : c.vocab <= 0) ||
        !(c.temperature > 0.0f) || c.activation_mode < RDCN_ACT_STORAGE || c.activation_mode > RDCN_ACT_F16 ||
        (c.parallel_branch != 0 && c.parallel_branch != 1) || (c.parallel_branch && c.attn_alpha == 0.0f) ||
        c.attn_alpha != c.attn_alpha || c.skip_beta != c.skip_beta)
        return RDCN_ERR_ARG;
    // ids in [0, vocab) (hashed: both 32-bit hash halves) must reach only existing rows
    const int64_t id_space = c.hashed ? ((int64_t)1 << 32) : c.vocab;
    if ((int64_t)c.qr_rows_q * (int64_t)c.qr_rows_r < id_space) return RDCN_ERR_SHAPE;
    const int64_t d = (int64_t)c.num_cat * c.emb_dim + c.num_dense;
    if (d <= 0) return RDCN_ERR_SHAPE;
    const int vec = c.dtype == RDCN_BF16 ? 8 : 4;
    if (c.emb_dim % vec || c.num_dense % vec || c.rank % vec || c.emb_dim > 256) return RDCN_ERR_UNSUPPORTED;
    const int n = c.attn_alpha != 0.0f ? 3 : 1;
    // sort keys and occurrence indices are 32-bit
    if ((int64_t)c.num_cat * (c.hashed ? 2 : 1) * ((int64_t)c.qr_rows_q + c.qr_rows_r) >= (int64_t)1 << 31)
        return RDCN_ERR_UNSUPPORTED;
    if (c.attn_alpha != 0.0f && c.rank > 1024) return RDCN_ERR_UNSUPPORTED;  // one sample's attention staged in LDS (<= 64 KiB)
    if (c.activation_mode != RDCN_ACT_STORAGE && c.dtype != RDCN_BF16) return RDCN_ERR_UNSUPPORTED;  // float storage is exact
    if (c.activation_mode != RDCN_ACT_STORAGE && c.parallel_branch) return RDCN_ERR_UNSUPPORTED;
    (void)n;

    rdcn_handle* h = new (std::nothrow) rdcn_handle();
    if (!h) return RDCN_ERR_HIP;
    h->cfg = c;
    h->d = d;
    h->attn = c.attn_alpha != 0.0f;
    h->par = c.parallel_branch != 0;
    h->n = h->attn ? (h->par ? 4 : 3) : 1;
    h->hr = h->par ? 2 * c.rank : c.rank;
    h->bf16 = c.dtype == RDCN_BF16;
    h->ids64 = c.id_type == RDCN_I64;
    h->split = c.activation_mode == RDCN_ACT_HILO;
    h->f16 = c.activation_mode == RDCN_ACT_F16;
    div_magic_host((uint32_t)c.qr_rows_r, h->magic, h->shift);
    if (hipMalloc((void**)&h->err, sizeof(int)) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return RDCN_ERR_HIP;
    }
    bool ok = hipMemset(h->err, 0, sizeof(int)) == hipSuccess && hipDeviceSynchronize() == hipSuccess;
    ok = ok && hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) == hipSuccess;  // default priority
    ok = ok && emb_static_scratch(&h->static_scratch) == hipSuccess;
    for (hipEvent_t* e : {&h->ev_pw, &h->ev_att, &h->ev_side[0], &h->ev_side[1], &h->ev_join})
        ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
    if (!ok) {
        (void)hipGetLastError();
        (void)rdcn_destroy(h);
        return RDCN_ERR_HIP;
    }
    *out = h;
    return RDCN_OK;
}

rdcn_status rdcn_destroy(rdcn_handle* h) {
    if (!h) return RDCN_OK;
    rdcn_status s = RDCN_OK;
    for (hipEvent_t e : h->prof_ev) (void)hipEventDestroy(e);
    for (hipEvent_t e : {h->ev_pw, h->ev_att, h->ev_side[0], h->ev_side[1], h->ev_join})
        if (e && hipEventDestroy(e) != hipSuccess) s = RDCN_ERR_HIP;
    if (h->side && hipStreamDestroy(h->side) != hipSuccess) s = RDCN_ERR_HIP;
    if (h->err && hipFree(h->err) != hipSuccess) s = RDCN_ERR_HIP;
    delete h;
    return s;
}

rdcn_status rdcn_dim(const rdcn_handle* h, int64_t* d) {
    if (!h || !d) return RDCN_ERR_ARG;
    *d = h->d;
    return RDCN_OK;
}

rdcn_status rdcn_workspace_bytes(const rdcn_handle* h, int64_t batch, size_t* saved_bytes, size_t* scratch_bytes) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (!saved_bytes || !scratch_bytes) return RDCN_ERR_ARG;
    *saved_bytes = saved_layout(h, batch).total;
    *scratch_bytes = std::max(scratch_layout(h, batch).total, fwd_scratch_layout(h).total);
    return RDCN_OK;
}

rdcn_status qr_embed_gather(rdcn_handle* h, int64_t batch, const void* ids, const int64_t* offsets,
                            const void* q_tables, const void* r_tables, const void* dense, void* x0, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    const rdcn_config& c = h->cfg;
    if ((offsets != nullptr) != (c.multi_hot != 0)) return RDCN_ERR_ARG;
    if (batch == 0) return RDCN_OK;
    GatherArgs a;
    if ((st = gather_args(h, batch, ids, offsets, q_tables, r_tables, dense, x0, a)) != RDCN_OK) return st;
    ProfScope ps(h, RDCN_KERNEL_GATHER, (hipStream_t)stream);
    return hip_status(launch_qr_gather(a, h->bf16, h->ids64, (hipStream_t)stream));
}

rdcn_status qr_quantize_tables(rdcn_handle* h, int64_t rows, const void* tables, int8_t* codes, float* params,
                               void* stream) {
    if (!h || rows < 0) return RDCN_ERR_ARG;
    if (rows >= ((int64_t)1 << 32)) return RDCN_ERR_UNSUPPORTED;
    if (rows == 0) return RDCN_OK;
    if (!tables || !codes || !params || !q8_aligned(h, codes, params)) return RDCN_ERR_ARG;
    ProfScope ps(h, RDCN_KERNEL_QUANTIZE, (hipStream_t)stream);
    return hip_status(launch_quantize_rows(rows, h->cfg.emb_dim, tables, codes, params, h->bf16, (hipStream_t)stream));
}

rdcn_status qr_embed_gather_q8(rdcn_handle* h, int64_t batch, const void* ids, const int64_t* offsets,
                               const int8_t* q_codes, const float* q_params, const int8_t* r_codes,
                               const float* r_params, const void* dense, void* x0, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if ((offsets != nullptr) != (h->cfg.multi_hot != 0)) return RDCN_ERR_ARG;
    if (batch == 0) return RDCN_OK;
    GatherArgs a;
    if ((st = gather_args(h, batch, ids, offsets, q_codes, r_codes, dense, x0, a)) != RDCN_OK) return st;
    if (h->cfg.num_cat > 0 && (!q_params || !r_params || !q8_aligned(h, q_codes, q_params) ||
                               !q8_aligned(h, r_codes, r_params)))
        return RDCN_ERR_ARG;
    a.q_params = q_params;
    a.r_params = r_params;
    ProfScope ps(h, RDCN_KERNEL_GATHER_Q8, (hipStream_t)stream);
    return hip_status(launch_qr_gather_q8(a, h->bf16, h->ids64, (hipStream_t)stream));
}

rdcn_status qr_embed_backward_workspace(const rdcn_handle* h, int64_t batch, int64_t nnz, size_t* scratch_bytes) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (!scratch_bytes || nnz < 0) return RDCN_ERR_ARG;
    if (!h->cfg.multi_hot && nnz != batch * h->cfg.num_cat) return RDCN_ERR_SHAPE;
    if (emb_pairs(nnz, h->cfg.hashed != 0) >= ((int64_t)1 << 31)) return RDCN_ERR_UNSUPPORTED;
    if (emb_fused_ok(h->cfg.qr_rows_q, h->cfg.qr_rows_r, h->cfg.emb_dim, h->cfg.hashed != 0)) {
        *scratch_bytes = 0;  // the one-kernel path needs no workspace
        return RDCN_OK;
    }
    const EmbedBwdLayout L =
        embed_bwd_layout(nnz, h->cfg.num_cat, h->cfg.qr_rows_q, h->cfg.qr_rows_r, h->cfg.emb_dim, h->cfg.multi_hot,
                         h->cfg.combine == RDCN_COMBINE_MUL, h->cfg.hashed != 0);
    *scratch_bytes = al(L.total);
    return RDCN_OK;
}

rdcn_status qr_embed_backward(rdcn_handle* h, int64_t batch, int64_t nnz, const void* ids, const int64_t* offsets,
                              const void* q_tables, const void* r_tables, const float* grad_x0,
                              float* grad_q_tables, float* grad_r_tables, void* scratch, size_t scratch_bytes,
                              void* stream) {
    size_t need = 0;
    rdcn_status st = qr_embed_backward_workspace(h, batch, nnz, &need);
    if (st != RDCN_OK) return st;
    const rdcn_config& c = h->cfg;
    if ((offsets != nullptr) != (c.multi_hot != 0)) return RDCN_ERR_ARG;
    if (batch == 0 || nnz == 0 || c.num_cat == 0) return RDCN_OK;
    if (!ids || !q_tables || !r_tables || !grad_x0 || !grad_q_tables || !grad_r_tables || (need > 0 && !scratch))
        return RDCN_ERR_ARG;
    if (need > 0 && (scratch_bytes < need || !aligned256(scratch))) return RDCN_ERR_WORKSPACE;
    if ((((uintptr_t)grad_x0) | ((uintptr_t)grad_q_tables) | ((uintptr_t)grad_r_tables)) & 15) return RDCN_ERR_ARG;
    EmbedBwdArgs a;
    a.batch = batch;
    a.nnz = nnz;
    a.d = h->d;
    a.F = c.num_cat;
    a.D = c.emb_dim;
    a.rows_q = c.qr_rows_q;
    a.m = (uint32_t)c.qr_rows_r;
    a.vocab = (uint64_t)c.vocab;
    a.combine = c.combine == RDCN_COMBINE_MUL ? 0 : 1;
    a.hashed = c.hashed;
    a.seed = c.hash_seed;
    a.ids = ids;
    a.offsets = offsets;
    a.q_tables = q_tables;
    a.r_tables = r_tables;
    a.grad_x0 = grad_x0;
    a.grad_q = grad_q_tables;
    a.grad_r = grad_r_tables;
    div_magic_host((uint32_t)c.num_cat, a.magic_f, a.shift_f);
    div_magic_host((uint32_t)c.qr_rows_q, a.magic_q, a.shift_q);
    a.magic_m = h->magic;
    a.shift_m = h->shift;
    hipStream_t s = (hipStream_t)stream;
    if (need == 0) {
        ProfScope ps(h, RDCN_KERNEL_EMB_FUSED, s);
        return hip_status(launch_emb_fused(a, h->bf16, h->ids64, s));
    }
    {
        ProfScope ps(h, RDCN_KERNEL_EMB_KEYS, s);
        RDCN_TRY(launch_emb_keys(a, h->ids64, scratch, s));
    }
    {
        ProfScope ps(h, RDCN_KERNEL_EMB_SORT, s);
        RDCN_TRY(launch_emb_sort(a, scratch, s));
    }
    ProfScope ps(h, RDCN_KERNEL_EMB_REDUCE, s);
    return hip_status(launch_emb_reduce(a, h->bf16, scratch, s));
}

// Once the backward has forked work onto the side stream, every return joins it back:
// nothing enqueued on the caller's stream afterwards can overlap work still running there.
struct SideJoin {
    rdcn_handle* h;
    hipStream_t s;
    bool forked;
    ~SideJoin() {
        if (forked && hipEventRecord(h->ev_join, h->side) == hipSuccess) (void)hipStreamWaitEvent(s, h->ev_join, 0);
    }
};

rdcn_status qr_embed_backward_static(rdcn_handle* h, int64_t batch, int64_t nnz, const void* ids,
                                     const int64_t* offsets, const void* q_tables, const void* r_tables,
                                     const float* grad_x0, float* grad_q_tables, float* grad_r_tables, void* stream) {
    size_t need = 0;
    rdcn_status st = qr_embed_backward_workspace(h, batch, nnz, &need);
    if (st != RDCN_OK) return st;
    if (need > RDCN_EMBED_STATIC_SCRATCH_BYTES) return RDCN_ERR_WORKSPACE;
    if (need > 0 && !h->static_scratch) return RDCN_ERR_HIP;
    return qr_embed_backward(h, batch, nnz, ids, offsets, q_tables, r_tables, grad_x0, grad_q_tables, grad_r_tables,
                             need > 0 ? h->static_scratch : nullptr, need, stream);
}

static rdcn_status check_weights(const rdcn_handle* h, const rdcn_weights* w) {
    if (!w) return RDCN_ERR_ARG;
    for (int l = 0; l < h->cfg.num_layers; ++l)
        if (!w->w_down[l] || !w->u[l] || !w->bias[l]) return RDCN_ERR_ARG;
    return RDCN_OK;
}

rdcn_status rdcn_forward(rdcn_handle* h, int64_t batch, const void* x0, const rdcn_weights* w, void* x_out,
                         void* saved, void* scratch, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if ((st = check_weights(h, w)) != RDCN_OK) return st;
    if (batch == 0) return RDCN_OK;
    if (!x0 || !x_out || !saved) return RDCN_ERR_ARG;
    if (!aligned256(saved)) return RDCN_ERR_WORKSPACE;
    const FwdScratchLayout FS = fwd_scratch_layout(h);
    if (FS.total > 0 && (!scratch || !aligned256(scratch))) return RDCN_ERR_WORKSPACE;
    if (h->f16) {  // the f16 copies of the weights use 16-byte vector accesses
        for (int l = 0; l < h->cfg.num_layers; ++l)
            if (!a16(w->w_down[l]) || !a16(w->u[l])) return RDCN_ERR_ARG;
    }
    hipStream_t s = (hipStream_t)stream;
    const rdcn_config& c = h->cfg;
    const int64_t B = batch, d = h->d, r = c.rank, nr = (int64_t)h->n * r;
    const SavedLayout S = saved_layout(h, B);
    char* sv = (char*)saved;
    void* w16 = FS.total ? (char*)scratch + FS.w16 : nullptr;  // f16 W_l (activation mode 2)
    void* u16 = FS.total ? (char*)scratch + FS.u16 : nullptr;  // f16 U_l
    const void* xcur = x0;        // x_l (hi plane when split, f16 in mode 2; x0 itself is bf16)
    const void* xcur2 = nullptr;  // lo plane of x_l when split (x0 is exact in bf16: none)
    for (int l = 0; l < c.num_layers; ++l) {
        const bool more = l + 1 < c.num_layers;
        const bool xf16 = h->f16 && l > 0;  // x_l held as f16
        void* P = sv + S.P[l];
        const int64_t hr = h->hr;
        // parallel branches: the plain branch's value V1^T x_l goes straight into the
        // first half of H; the attention branch's [v2|q|k] into P as usual
        const int64_t pr = h->par ? 3 * r : nr;  // width of P
        const char* wv = (const char*)w->w_down[l] + (h->par ? r * d * (int64_t)eb(h) : 0);
        if (h->f16) {  // this layer's weights as f16 operands (W only when x_l is f16)
            if (xf16) RDCN_TRY(launch_bf16_to_f16(w->w_down[l], w16, nr * d, h->err, s));
            RDCN_TRY(launch_bf16_to_f16(w->u[l], u16, d * hr, h->err, s));
        }
        if (h->par) {
            GemmArgs g{};
            g.M = B; g.N = r; g.K = d;
            g.a = xcur; g.lda = d;
            g.b = w->w_down[l]; g.ldb = d;
            g.epi = EPI_STORE; g.scale = 1.0f;
            g.c = sv + S.H[l]; g.ldc = hr;
            ProfScope ps(h, RDCN_KERNEL_FWD_DOWN_GEMM, s);
            RDCN_TRY(launch_gemm(g, plan_gemm(B, r, d, h->bf16, false), h->bf16, s));
        }
        GemmArgs g{};
        g.M = B; g.N = pr; g.K = d;
        g.a = xcur; g.a2 = xcur2; g.lda = d;
        g.b = xf16 ? w16 : wv; g.ldb = d;
        g.ops_f16 = xf16;
        g.epi = h->attn ? EPI_STORE_F32 : EPI_STORE; g.scale = 1.0f;
        g.c = P; g.ldc = pr;
        g.err = h->err;
        if (!h->attn && (h->split || h->f16)) {  // v as hi + lo, or its f16 copy, for the up projection
            g.c2 = sv + S.P2[l];
            g.c2_kind = h->f16 ? C2_F16 : C2_LO;
        }
        {
            ProfScope ps(h, RDCN_KERNEL_FWD_DOWN_GEMM, s);
            RDCN_TRY(launch_gemm(g, plan_gemm(B, pr, d, h->bf16, false), h->bf16, s));
        }
        const void* hsrc = P;
        const void* hsrc2 = h->split ? g.c2 : nullptr;
        int64_t ldh = nr;
        float scale = c.skip_beta;
        if (h->f16 && !h->attn) hsrc = g.c2;  // the f16 copy of v
        if (h->attn) {
            void* H = sv + S.H[l];
            void* H2 = (h->split || h->f16) ? (void*)(sv + S.H2[l]) : nullptr;
            void* Ha = (char*)H + (h->par ? r * (int64_t)eb(h) : 0);  // attention output columns of H
            ProfScope ps(h, RDCN_KERNEL_FWD_ATTENTION, s);
            RDCN_TRY(launch_attn_fwd(B, (int)r, c.attn_alpha, c.skip_beta, c.temperature, P, pr, Ha, H2, h->f16, hr,
                                     (float*)(sv + S.A[l]), h->err, h->bf16, s));
            hsrc = h->f16 ? H2 : H;
            hsrc2 = h->split ? H2 : nullptr;
            ldh = hr;
            scale = 1.0f;
        }
        void* xnext = more ? (void*)(sv + S.X[l]) : x_out;
        GemmArgs u{};
        u.M = B; u.N = d; u.K = hr;
        u.a = hsrc; u.a2 = hsrc2; u.lda = ldh;
        u.b = h->f16 ? u16 : w->u[l]; u.ldb = hr;
        u.ops_f16 = h->f16;
        u.epi = EPI_CROSS; u.scale = scale;
        u.c = xnext; u.ldc = d;
        u.err = h->err;
        if (more && (h->split || h->f16)) {  // x_{l+1}: hi + lo pair, or f16 with a bf16 copy
            u.c2 = sv + S.X2[l];
            u.c2_kind = h->f16 ? C2_BF16 : C2_LO;
            u.c_f16 = h->f16;
        }
        u.bias = w->bias[l]; u.x0 = x0; u.xl = xcur; u.xl2 = xcur2; u.xl_f16 = xf16;
        u.t_out = sv + S.T[l]; u.ldx = d;
        {
            ProfScope ps(h, RDCN_KERNEL_FWD_UP_GEMM, s);
            RDCN_TRY(launch_gemm(u, plan_gemm(B, d, hr, h->bf16, false), h->bf16, s));
        }
        xcur = xnext;
        xcur2 = h->split ? u.c2 : nullptr;
    }
    return RDCN_OK;
}

rdcn_status rdcn_backward(rdcn_handle* h, int64_t batch, const void* x0, const rdcn_weights* w, const void* saved,
                          const void* grad_out, float* grad_x0, const rdcn_weights* grads, void* scratch,
                          void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if ((st = check_weights(h, w)) != RDCN_OK) return st;
    if ((st = check_weights(h, grads)) != RDCN_OK) return st;
    const rdcn_config& c = h->cfg;
    hipStream_t s = (hipStream_t)stream;
    const int64_t B = batch, d = h->d, r = c.rank, nr = (int64_t)h->n * r;
    if (batch == 0) {  // gradients of an empty batch are zero
        for (int l = 0; l < c.num_layers; ++l) {
            RDCN_TRY(launch_fill_zero((float*)grads->w_down[l], nr * d, s));
            RDCN_TRY(launch_fill_zero((float*)grads->u[l], d * (int64_t)h->hr, s));
            RDCN_TRY(launch_fill_zero((float*)grads->bias[l], d, s));
        }
        return RDCN_OK;
    }
    if (!x0 || !saved || !grad_out || !grad_x0 || !scratch) return RDCN_ERR_ARG;
    if (!aligned256(saved) || !aligned256(scratch)) return RDCN_ERR_WORKSPACE;
    const SavedLayout S = saved_layout(h, B);
    const ScratchLayout W = scratch_layout(h, B);
    const char* sv = (const char*)saved;
    char* sc = (char*)scratch;
    float* g = (float*)(sc + W.g);
    float* gh = (float*)(sc + W.gh);
    float* splitk = (float*)(sc + W.splitk);
    const bool use_side = h->side_enabled;
    hipStream_t side = use_side ? h->side : s;
    SideJoin join{h, s, false};

    // Main stream: pointwise -> gh -> attention -> gx, the chain from one layer's
    // gradient to the next. Side stream, once the layer's attention is done: the bias
    // column sums and the weight gradients gU and gW (with their split-K reductions),
    // which nothing later in the backward reads; they overlap gx and the next layer's
    // pointwise and gh (started earlier, they slow the attention more than they gain;
    // layer 0, the last, starts its bias sums and gU after its pointwise kernel).
    for (int l = c.num_layers - 1; l >= 0; --l) {
        const bool top = l == c.num_layers - 1;
        const int par = l & 1;
        void* gt = sc + W.gt[par];
        void* gP = sc + W.gP[par];
        float* part = (float*)(sc + W.part[par]);
        // this parity's copies were last read by the side stream's work of layer l + 2
        if (use_side && l + 2 < c.num_layers) RDCN_TRY(hipStreamWaitEvent(s, h->ev_side[par], 0));
        const void* gin = top ? grad_out : (const void*)g;
        const void* P = sv + S.P[l];
        // x_l as the weight gradient's bf16 operand (the hi plane, or the bf16 copy of an f16 x_l)
        const void* xl = l == 0 ? x0 : (const void*)(sv + (h->f16 ? S.X2[l - 1] : S.X[l - 1]));
        // gt = g * x0, grad_x0 (+)= g * t_l, bias partials
        {
            ProfScope ps(h, RDCN_KERNEL_BWD_POINTWISE, s);
            RDCN_TRY(launch_bwd_pointwise(B, d, gin, !top, x0, sv + S.T[l], grad_x0, top, gt, part, h->bf16, s));
        }
        const void* hsrc = h->attn ? (const void*)(sv + S.H[l]) : P;
        const int64_t hr = h->hr;
        const int64_t ldh = h->attn ? hr : nr;
        const float hscale = h->attn ? 1.0f : c.skip_beta;
        const int64_t e = (int64_t)eb(h);
        // bias sums and gU on the side stream
        auto side_bias_gu = [&]() -> rdcn_status {
            {
                ProfScope ps(h, RDCN_KERNEL_BWD_BIAS, side);
                RDCN_TRY(launch_colsum(part, W.nrb, d, (float*)grads->bias[l], side));
            }
            // gU = gt^T h      [d, hr], K = batch
            {
                GemmArgs g1{};
                g1.M = d; g1.N = hr; g1.K = B;
                g1.a = gt; g1.lda = d; g1.a_kstrided = true;
                g1.b = hsrc; g1.ldb = ldh; g1.b_kstrided = true;
                g1.scale = hscale;
                RDCN_TRY(gemm_weight_grad(h, RDCN_KERNEL_BWD_GU_GEMM, g1, (float*)grads->u[l], splitk, side,
                                          bwd_split_blocks(g1.M, g1.N, g1.K)));
            }
            return RDCN_OK;
        };
        // Layer 0 forks its bias sums and gU right after the pointwise kernel: nothing
        // follows its gx on the main stream, so side work left until after the attention
        // would run alone while the main stream waits to join.
        if (l == 0) {
            if (use_side) {
                RDCN_TRY(hipEventRecord(h->ev_pw, s));
                RDCN_TRY(hipStreamWaitEvent(side, h->ev_pw, 0));
                join.forked = true;
            }
            if ((st = side_bias_gu()) != RDCN_OK) return st;
        }
        // gh = gt U         [B, hr]; with parallel branches the plain branch's part is its
        // value gradient and goes straight into the first columns of gP
        if (h->par) {
            GemmArgs g2{};
            g2.M = B; g2.N = r; g2.K = d;
            g2.a = gt; g2.lda = d;
            g2.b = w->u[l]; g2.ldb = hr; g2.b_kstrided = true;
            g2.epi = EPI_STORE; g2.scale = 1.0f; g2.c = gP; g2.ldc = nr;
            ProfScope ps(h, RDCN_KERNEL_BWD_GH_GEMM, s);
            RDCN_TRY(launch_gemm(g2, plan_gemm(B, r, d, h->bf16, false), h->bf16, s));
        }
        {
            GemmArgs g2{};
            g2.M = B; g2.N = r; g2.K = d;
            g2.a = gt; g2.lda = d;
            g2.b = (const char*)w->u[l] + (h->par ? r * e : 0); g2.ldb = hr; g2.b_kstrided = true;
            if (h->attn) {
                g2.epi = EPI_STORE_F32; g2.scale = 1.0f; g2.c = gh; g2.ldc = r;
            } else {
                g2.epi = EPI_STORE; g2.scale = c.skip_beta; g2.c = gP; g2.ldc = nr;  // gv = beta * gh
            }
            ProfScope ps(h, RDCN_KERNEL_BWD_GH_GEMM, s);
            RDCN_TRY(launch_gemm(g2, plan_gemm(B, r, d, h->bf16, false), h->bf16, s));
        }
        if (h->attn) {
            const int64_t pr = h->par ? 3 * r : nr;
            ProfScope ps(h, RDCN_KERNEL_BWD_ATTENTION, s);
            RDCN_TRY(launch_attn_bwd(B, (int)r, c.attn_alpha, c.skip_beta, c.temperature, P, pr,
                                     (const float*)(sv + S.A[l]), gh, r, (char*)gP + (h->par ? r * e : 0), nr,
                                     h->bf16, s));
        }
        if (use_side) {
            RDCN_TRY(hipEventRecord(h->ev_att, s));
            RDCN_TRY(hipStreamWaitEvent(side, h->ev_att, 0));
            join.forked = true;
        }
        if (l > 0 && (st = side_bias_gu()) != RDCN_OK) return st;
        // gW = gP^T x_l    [n r, d], K = batch
        {
            GemmArgs g3{};
            g3.M = nr; g3.N = d; g3.K = B;
            g3.a = gP; g3.lda = nr; g3.a_kstrided = true;
            g3.b = xl; g3.ldb = d; g3.b_kstrided = true;
            g3.scale = 1.0f;
            RDCN_TRY(gemm_weight_grad(h, RDCN_KERNEL_BWD_GW_GEMM, g3, (float*)grads->w_down[l], splitk, side,
                                      bwd_split_blocks(g3.M, g3.N, g3.K)));
        }
        if (use_side) RDCN_TRY(hipEventRecord(h->ev_side[par], side));
        // g_l = g_{l+1} + gP W   (layer 0: grad_x0 += g_1 + gP W)
        {
            GemmArgs g4{};
            g4.M = B; g4.N = d; g4.K = nr;
            g4.a = gP; g4.lda = nr;
            g4.b = w->w_down[l]; g4.ldb = d; g4.b_kstrided = true;
            g4.scale = 1.0f;
            g4.gin = gin; g4.gin_f32 = !top; g4.ldx = d;
            g4.epi = l == 0 ? EPI_RESID_X0 : EPI_RESID;
            g4.c = l == 0 ? (void*)grad_x0 : (void*)g; g4.ldc = d;
            ProfScope ps(h, RDCN_KERNEL_BWD_GX_GEMM, s);
            RDCN_TRY(launch_gemm(g4, plan_gemm(B, d, nr, h->bf16, false), h->bf16, s));
        }
    }
    // join: the side stream's last work (layer 0) completes before anything later on `s`
    if (use_side) {
        join.forked = false;
        RDCN_TRY(hipStreamWaitEvent(s, h->ev_side[0], 0));
    }
    return RDCN_OK;
}

rdcn_status rdcn_head_configure(rdcn_handle* h, const rdcn_head_config* cfg) {
    if (!h || !cfg) return RDCN_ERR_ARG;
    const rdcn_head_config& c = *cfg;
    if (c.num_hidden < 1 || c.num_hidden > RDCN_HEAD_MAX_HIDDEN || (c.gated != 0 && c.gated != 1) ||
        c.num_buckets < 1 || c.num_buckets > 65536 || !std::isfinite(c.bucket_lo) || !std::isfinite(c.bucket_step) ||
        !(c.bucket_step > 0.0f))
        return RDCN_ERR_ARG;
    for (int l = 0; l < c.num_hidden; ++l)
        if (c.hidden[l] <= 0 || c.hidden[l] % 8) return RDCN_ERR_ARG;
    if (!h->bf16) return RDCN_ERR_UNSUPPORTED;
    if (h->cfg.batch_max > (int64_t)65535 * 64) return RDCN_ERR_UNSUPPORTED;  // column-sum chunks per launch
    h->head = c;
    for (int l = c.num_hidden; l < RDCN_HEAD_MAX_HIDDEN; ++l) h->head.hidden[l] = 0;
    h->head_on = true;
    return RDCN_OK;
}

rdcn_status rdcn_head_workspace_bytes(const rdcn_handle* h, int64_t batch, size_t* saved_bytes,
                                      size_t* scratch_bytes) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (!h->head_on) return RDCN_ERR_ARG;
    if (!saved_bytes || !scratch_bytes) return RDCN_ERR_ARG;
    *saved_bytes = head_saved_layout(h, batch).total;
    *scratch_bytes = head_scratch_layout(h, batch).total;
    return RDCN_OK;
}

rdcn_status rdcn_head_forward(rdcn_handle* h, int64_t batch, const void* x, const float* e_cal,
                              const rdcn_head_weights* w, float* y_logit, float* y_cal, void* saved, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (!h->head_on) return RDCN_ERR_ARG;
    if ((st = check_head_weights(h, w)) != RDCN_OK) return st;
    if (batch == 0) return RDCN_OK;
    if (!x || !a16(x) || !e_cal || !y_logit || !y_cal || !saved) return RDCN_ERR_ARG;
    if (!aligned256(saved)) return RDCN_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    const rdcn_head_config& c = h->head;
    const int64_t B = batch;
    const HeadSaved S = head_saved_layout(h, B);
    char* sv = (char*)saved;
    for (int l = 0; l < c.num_hidden; ++l) {
        const int64_t nin = head_in(h, l), nout = c.hidden[l];
        // layer 0 reads the bf16 input, the others the f16 copy of a_{l-1}
        const void* in = l == 0 ? x : (const void*)(sv + S.A16[l - 1]);
        float* sl = c.gated ? (float*)(sv + S.S[l]) : nullptr;
        if (c.gated) {
            ProfScope ps(h, RDCN_KERNEL_HEAD_GATE, s);
            RDCN_TRY(launch_gate_logit(B, (int)nin, in, l > 0, nin, w->gate_w[l], w->gate_b[l], sl, s));
        }
        GemmArgs g{};
        g.M = B; g.N = nout; g.K = nin;
        g.a = in; g.lda = nin;
        g.b = w->w[l]; g.ldb = nin;
        if (l > 0) {
            g.b = sv + S.W16;
            g.ops_f16 = true;
            RDCN_TRY(launch_bf16_to_f16(w->w[l], sv + S.W16, nout * nin, h->err, s));
        }
        g.epi = EPI_MLP_FWD; g.scale = 1.0f;
        g.bias = w->b[l];
        g.rowv = sl;
        g.c = sv + S.A[l]; g.ldc = nout;
        g.c2 = sv + S.A16[l]; g.c2_kind = C2_F16;
        g.err = h->err;
        ProfScope ps(h, RDCN_KERNEL_HEAD_FWD_GEMM, s);
        RDCN_TRY(launch_gemm(g, plan_gemm(B, nout, nin, true, false), true, s));
    }
    const int L = c.num_hidden;
    ProfScope ps(h, RDCN_KERNEL_HEAD_OUT, s);
    return hip_status(launch_head_out(B, c.hidden[L - 1], sv + S.A16[L - 1], w->w_out, w->b_out,
                                      cal_args(h, w, e_cal), (float*)(sv + S.Y), y_logit, y_cal, s));
}

rdcn_status rdcn_head_logloss(rdcn_handle* h, int64_t batch, const float* y_cal, const float* labels, float scale,
                              float* loss, float* grad, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (batch == 0) return RDCN_OK;
    if (!y_cal || !labels || !std::isfinite(scale)) return RDCN_ERR_ARG;
    ProfScope ps(h, RDCN_KERNEL_HEAD_LOSS, (hipStream_t)stream);
    return hip_status(launch_logloss(batch, y_cal, labels, scale, loss, grad, (hipStream_t)stream));
}

rdcn_status rdcn_head_backward(rdcn_handle* h, int64_t batch, const void* x, const float* e_cal,
                               const rdcn_head_weights* w, const void* saved, const float* grad_ycal, void* grad_x,
                               float* grad_e, const rdcn_head_weights* grads, void* scratch, void* stream) {
    rdcn_status st = check_batch(h, batch);
    if (st != RDCN_OK) return st;
    if (!h->head_on) return RDCN_ERR_ARG;
    if ((st = check_head_weights(h, w)) != RDCN_OK) return st;
    if ((st = check_head_weights(h, grads)) != RDCN_OK) return st;
    if (!scratch || !aligned256(scratch)) return RDCN_ERR_WORKSPACE;
    if (batch > 0) {
        if (!x || !a16(x) || !e_cal || !saved || !grad_ycal || !grad_x || !a16(grad_x) || !grad_e)
            return RDCN_ERR_ARG;
        if (!aligned256(saved)) return RDCN_ERR_WORKSPACE;
    }
    hipStream_t s = (hipStream_t)stream;
    const rdcn_head_config& c = h->head;
    const int64_t B = batch;
    const int L = c.num_hidden;
    const HeadSaved S = head_saved_layout(h, B);
    const HeadScratch W = head_scratch_layout(h, B);
    const char* sv = (const char*)saved;
    char* sc = (char*)scratch;
    float* gy = (float*)(sc + W.gy);
    float* colpart = (float*)(sc + W.colpart);
    auto gs_of = [&](int l) { return (float*)(sc + W.gs + (size_t)l * al((size_t)B * 4)); };
    VecSums sums{};  // the scalar gradients, summed in one launch at the end
    auto add_sum = [&](const float* x, void* out) {
        sums.x[sums.n] = x;
        sums.out[sums.n] = (float*)out;
        ++sums.n;
    };
    auto colsum = [&](int64_t n, const void* X, int64_t ldx, ColType xt, const float* wgt, void* out) -> hipError_t {
        ProfScope ps(h, RDCN_KERNEL_HEAD_COLSUM, s);
        return launch_colsum_w(B, n, X, ldx, xt, wgt, colpart, (float*)out, s);
    };
    // the top layer's activations as the forward's logit read them (f16)
    const void* aL = B > 0 ? (const void*)(sv + S.A16[L - 1]) : nullptr;
    int cur = 0;
    {
        ProfScope ps(h, RDCN_KERNEL_HEAD_OUT_BWD, s);
        RDCN_TRY(launch_head_out_bwd(B, c.hidden[L - 1], aL, c.gated && B > 0 ? (const float*)(sv + S.S[L - 1]) : nullptr,
                                     w->w_out, B > 0 ? (const float*)(sv + S.Y) : nullptr, cal_args(h, w, e_cal),
                                     grad_ycal, grad_e, gy, sc + W.G[cur], gs_of(L - 1), s));
    }
    RDCN_TRY(colsum(c.hidden[L - 1], aL, c.hidden[L - 1], COL_F16, gy, grads->w_out));
    RDCN_TRY(colsum(c.num_buckets, grad_e, c.num_buckets, COL_F32, nullptr, grads->cal_w));
    add_sum(gy, grads->b_out);
    add_sum(grad_ycal, grads->cal_b);
    for (int l = L - 1; l >= 0; --l) {
        const int64_t nin = head_in(h, l), nout = c.hidden[l];
        const void* in = l == 0 ? x : (const void*)(sv + S.A[l - 1]);
        const void* G = sc + W.G[cur];
        const float* gsl = gs_of(l);
        RDCN_TRY(colsum(nout, G, nout, COL_BF16, nullptr, grads->b[l]));
        if (c.gated) {
            // the gate logit's input as the forward read it (bf16 x, f16 a_{l-1})
            if (l == 0) RDCN_TRY(colsum(nin, in, nin, COL_BF16, gsl, grads->gate_w[l]));
            else RDCN_TRY(colsum(nin, sv + S.A16[l - 1], nin, COL_F16, gsl, grads->gate_w[l]));
            add_sum(gsl, grads->gate_b[l]);
        }
        {
            GemmArgs g{};
            g.M = nout; g.N = nin; g.K = B;
            g.a = G; g.lda = nout; g.a_kstrided = true;
            g.b = in; g.ldb = nin; g.b_kstrided = true;
            g.scale = 1.0f;
            RDCN_TRY(gemm_weight_grad(h, RDCN_KERNEL_HEAD_GW_GEMM, g, (float*)grads->w[l], (float*)(sc + W.splitk), s));
        }
        GemmArgs g{};
        g.M = B; g.N = nin; g.K = nout;
        g.a = G; g.lda = nout;
        g.b = w->w[l]; g.ldb = nin; g.b_kstrided = true;
        g.epi = EPI_MLP_BWD; g.scale = 1.0f;
        if (c.gated) {
            g.colv = w->gate_w[l];
            g.rowv = gsl;
        }
        const GemmPlan p = plan_gemm(B, nin, nout, true, false);
        if (l > 0) {
            g.act = sv + S.A[l - 1]; g.ldx = nin;
            g.c = sc + W.G[1 - cur]; g.ldc = nin;
            if (c.gated) {
                g.rowg = (const float*)(sv + S.S[l - 1]);
                g.rowpart = (float*)(sc + W.rowpart);
            }
        } else {
            g.c = grad_x; g.ldc = nin;
        }
        {
            ProfScope ps(h, RDCN_KERNEL_HEAD_GX_GEMM, s);
            RDCN_TRY(launch_gemm(g, p, true, s));
        }
        if (l > 0 && c.gated) {
            ProfScope ps(h, RDCN_KERNEL_HEAD_GATE_BWD, s);
            RDCN_TRY(launch_gate_finalize(B, (int)gemm_tiles_n(nin, p), (const float*)(sc + W.rowpart),
                                          (const float*)(sv + S.S[l - 1]), gs_of(l - 1), s));
        }
        cur = 1 - cur;
    }
    ProfScope ps(h, RDCN_KERNEL_HEAD_COLSUM, s);
    return hip_status(launch_vec_sums(B, sums, s));
}

rdcn_status rdcn_profile_start(rdcn_handle* h, int32_t max_launches, uint32_t kernel_mask) {
    if (!h || max_launches < 0) return RDCN_ERR_ARG;
    for (hipEvent_t e : h->prof_ev) (void)hipEventDestroy(e);
    h->prof_ev.clear();
    h->prof_kind.clear();
    h->prof_used = 0;
    h->prof_ev.resize(2 * (size_t)max_launches);
    // timing-only events: without the system-scope fence (cache write-back and
    // invalidation at every record) the timed kernel starts as it would untimed
    for (auto& e : h->prof_ev)
        if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return RDCN_ERR_HIP;
    h->prof_kind.reserve(max_launches);
    h->prof_mask = kernel_mask;
    h->prof_on = true;
    return RDCN_OK;
}

rdcn_status rdcn_profile_stop(rdcn_handle* h, double* ms, int64_t* launches) {
    if (!h || !ms || !launches) return RDCN_ERR_ARG;
    h->prof_on = false;
    for (int k = 0; k < RDCN_KERNEL_COUNT; ++k) {
        ms[k] = 0.0;
        launches[k] = 0;
    }
    rdcn_status st = RDCN_OK;
    for (size_t i = 0; i < h->prof_used; ++i) {
        if (hipEventSynchronize(h->prof_ev[2 * i + 1]) != hipSuccess) {
            st = RDCN_ERR_HIP;
            break;
        }
        float t = 0.f;
        if (hipEventElapsedTime(&t, h->prof_ev[2 * i], h->prof_ev[2 * i + 1]) != hipSuccess) {
            st = RDCN_ERR_HIP;
            break;
        }
        ms[h->prof_kind[i]] += t;
        launches[h->prof_kind[i]] += 1;
    }
    h->prof_used = 0;
    h->prof_kind.clear();
    return st;
}

rdcn_status rdcn_check_device_errors(rdcn_handle* h, void* stream) {
    if (!h) return RDCN_ERR_ARG;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return RDCN_ERR_HIP;
    int v = 0;
    if (hipMemcpy(&v, h->err, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess) return RDCN_ERR_HIP;
    if (v != 0) {
        const int zero = 0;
        if (hipMemcpy(h->err, &zero, sizeof(int), hipMemcpyHostToDevice) != hipSuccess) return RDCN_ERR_HIP;
        return (v & 1) ? RDCN_ERR_INDEX : RDCN_ERR_RANGE;
    }
    return RDCN_OK;
}

rdcn_status rdcn_set_side_stream(rdcn_handle* h, int32_t enable) {
    if (!h || (enable != 0 && enable != 1)) return RDCN_ERR_ARG;
    h->side_enabled = enable != 0;
    return RDCN_OK;
}

}  // extern "C"
