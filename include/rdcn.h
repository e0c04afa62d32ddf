/*
 * rdcn.h -- C ABI of the MI355X (gfx950) Residual-DCN + QR-embedding library (librdcn.so).
 *
 * The library computes, on one GPU, the forward and backward pass of the
 * interaction stack of LiRank (Borisyuk et al., KDD'24, arXiv 2402.06859):
 *
 *   x0      = [ emb_0 | ... | emb_{F-1} | dense ]                  (qr_embed_gather)
 *   emb_f   = pool over the bag of feature f of  Q_f[id / m] (op) R_f[id mod m]
 *   x_{l+1} = x0 * (U_l h_l + b_l) + x_l,   l = 0 .. L-1          (rdcn_forward)
 *   h_l     = beta * v + alpha * softmax_j(q_i k_j / tau) v,   [v; q; k] = W_l x_l
 *
 * and the gradients of a scalar loss given dLoss/dx_L (rdcn_backward,
 * qr_embed_backward). Paper passages:
 *   - QR split, per-feature quotient/remainder tables, sum or product combine:
 *     section "Model Dictionary Compression".
 *   - embedding look-ups replacing one-hot inputs, concatenated with dense
 *     features: section "Residual DCN" (first paragraph) and appendix
 *     "Feed Ranking Sparse ID features".
 *   - low-rank DCNv2 cross layer (two skinny matrices U, V): section
 *     "Residual DCN", first paragraph.
 *   - attention low-rank cross net (value/query/key copies of the low-rank
 *     map, attention score matrix between the low-rank maps, temperature)
 *     and the skip connection: section "Residual DCN", second paragraph. The
 *     paper describes this layer in prose only; this library reads it as
 *     attention over the r low-rank coordinates of one sample (an r x r score
 *     matrix per sample), with h = beta*v + alpha*o.
 *
 * Conventions
 *   - All tensors are dense row-major. Device pointers unless stated.
 *   - The caller allocates and frees every device buffer (inputs, weights,
 *     outputs, gradients, saved activations, scratch). The library allocates
 *     no device memory after rdcn_create (which allocates one small error word)
 *     and never frees caller memory.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the
 *     default stream). Arguments are validated on the host before anything is
 *     launched; on error nothing is launched.
 *   - A handle must not be used by two host threads at once.
 *   - No exception or abort crosses this ABI: every function returns an
 *     rdcn_status.
 */
#ifndef RDCN_H
#define RDCN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rdcn_status {
    RDCN_OK = 0,
    RDCN_ERR_ARG = 1,          /* null pointer, negative size, unknown enum value */
    RDCN_ERR_SHAPE = 2,        /* inconsistent sizes (batch > batch_max, rows_q * m < vocab, ...) */
    RDCN_ERR_INDEX = 3,        /* an id outside [0, vocab) was met on the device */
    RDCN_ERR_UNSUPPORTED = 4,  /* valid but not supported here (see rdcn_create) */
    RDCN_ERR_WORKSPACE = 5,    /* a workspace or buffer argument is too small */
    RDCN_ERR_HIP = 6,          /* a HIP runtime call or kernel launch failed */
    RDCN_ERR_RANGE = 7         /* an activation kept as f16 (activation mode 2, or a head's
                                  hidden activations) or an f16 weight copy was beyond the
                                  f16 range (|x| >= 65520) and became infinite */
} rdcn_status;

typedef enum rdcn_dtype { RDCN_F32 = 0, RDCN_BF16 = 1 } rdcn_dtype;
typedef enum rdcn_idtype { RDCN_I32 = 0, RDCN_I64 = 1 } rdcn_idtype;
typedef enum rdcn_combine { RDCN_COMBINE_MUL = 0, RDCN_COMBINE_SUM = 1 } rdcn_combine;

/*
 * Precision of the activations the projections read (bf16 models; float models
 * keep everything in float). The paper fixes no precision for the cross stack;
 * deep attention stacks whose softmax ends close to one-hot amplify any rounding of
 * x_l and h, so the library offers three ways to hold them:
 *   RDCN_ACT_STORAGE: x_l and h in bf16, the storage type (one bf16 MFMA pass each)
 *   RDCN_ACT_HILO:    x_l (l >= 1) and h as bf16 hi + lo pairs whose sum carries about
 *                     16 significant bits; the down and up projections run two bf16
 *                     MFMA passes over them against the exact bf16 weights
 *   RDCN_ACT_F16:     x_l (l >= 1) and h in f16 (11 significant bits; |x| < 65520, else
 *                     RDCN_ERR_RANGE is flagged); the down (l >= 1) and up projections
 *                     run one f16 MFMA pass against f16 copies of the weights that
 *                     rdcn_forward makes in its scratch (bf16 weights of magnitude
 *                     >= 2^-17 convert exactly); bf16 copies of x_l and h feed the
 *                     weight gradients
 */
typedef enum rdcn_act_mode { RDCN_ACT_STORAGE = 0, RDCN_ACT_HILO = 1, RDCN_ACT_F16 = 2 } rdcn_act_mode;

#define RDCN_MAX_LAYERS 16

/*
 * Model and batch description. d = num_cat * emb_dim + num_dense is derived.
 * n = 3 projections per layer (value, query, key) when attn_alpha != 0, else 1;
 * n = 4 with parallel branches (plain value, attention value, query, key).
 * hr = 2r with parallel branches, else r: the width of the up projection's input.
 */
typedef struct rdcn_config {
    int64_t batch_max;    /* largest batch any call will pass */
    int32_t num_cat;      /* F: categorical features (>= 0) */
    int32_t emb_dim;      /* D: embedding dimension (> 0) */
    int32_t num_dense;    /* Nd: dense features (>= 0) */
    int32_t rank;         /* r: low-rank dimension (> 0) */
    int32_t num_layers;   /* L: cross layers (1 .. RDCN_MAX_LAYERS) */
    int32_t qr_rows_q;    /* rows of every quotient table */
    int32_t qr_rows_r;    /* m: rows of every remainder table, and the QR divisor */
    int32_t combine;      /* rdcn_combine: how the two rows are aggregated */
    int32_t multi_hot;    /* 0: one id per (sample, feature); 1: CSR bags, sum pooling */
    int32_t id_type;      /* rdcn_idtype of the id array */
    int32_t dtype;        /* rdcn_dtype of tables, dense, x0, activations and weights */
    int32_t activation_mode; /* rdcn_act_mode; modes 1 and 2 need a bf16 model without
                                parallel branches */
    int64_t vocab;        /* V: valid ids are [0, V); requires qr_rows_q * qr_rows_r >= V */
    float attn_alpha;     /* alpha: weight of the attention path (0 = plain low-rank DCNv2) */
    float skip_beta;      /* beta: weight of the skip (value) path */
    float temperature;    /* tau > 0: scores are q_i k_j / tau */
    int32_t parallel_branch; /* 0 or 1 (needs attn_alpha != 0): a plain low-rank cross net and the
                                attention low-rank cross net run side by side with their own
                                weights (section "Residual DCN", last sentences of the second
                                paragraph): t = U1 V1^T x + U2 (beta v2 + alpha A v2) + b */
    int32_t hashed;       /* 0 or 1: hashed front-end (appendix "Vocabulary Compression"): every
                             raw id is hashed with MurmurHash64A (its 8 little-endian bytes,
                             seed hash_seed); the low 32 bits B and the high 32 bits C each
                             index their own QR table pair, and the two combined rows are
                             summed. Tables become [F, 2, rows, D] (pair 0 for B, 1 for C),
                             vocab must be 0 (every id is valid), and qr_rows_q * m must
                             reach 2^32 */
    int32_t reserved2;    /* must be 0 */
    uint64_t hash_seed;   /* seed of the hashed front-end */
} rdcn_config;

/*
 * Per-layer weight pointers (entries at index >= num_layers are ignored).
 *   w_down[l] : [n*r, d]  rows 0..r-1 = V_l^T (value), r..2r-1 = Q_l^T, 2r..3r-1 = K_l^T;
 *                         with parallel branches V1^T (plain branch), V2^T, Q^T, K^T
 *   u[l]      : [d, hr]   up projection U_l ([U1 | U2] with parallel branches)
 *   bias[l]   : [d]       b_l
 * Weights are in the storage dtype; gradients use the same struct with float pointers.
 */
typedef struct rdcn_weights {
    void* w_down[RDCN_MAX_LAYERS];
    void* u[RDCN_MAX_LAYERS];
    void* bias[RDCN_MAX_LAYERS];
} rdcn_weights;

typedef struct rdcn_handle rdcn_handle;

/*
 * Validate `cfg` and create a handle (host metadata plus one device error word
 * on the current device). The configuration is the paper's statement of the
 * model: categorical ids QR-hashed into per-feature quotient and remainder
 * tables (section "Model Dictionary Compression"), their embeddings
 * concatenated with the dense features (appendix "Feed Ranking Sparse ID
 * features"), and a stack of num_layers Residual DCN layers of rank r with the
 * attention term and skip weight (section "Residual DCN").
 * Returns RDCN_ERR_ARG for null pointers or values out
 * of range, RDCN_ERR_SHAPE if qr_rows_q * qr_rows_r < vocab, and
 * RDCN_ERR_UNSUPPORTED when a bf16 model has emb_dim, num_dense or rank not a
 * multiple of 8 (fp32: multiple of 4), which the vector loads need, when
 * emb_dim > 256, when the attention term is on with rank > 1024 (one sample's
 * attention operands are staged in 64 KiB of LDS), or when F * (qr_rows_q + m)
 * does not fit the 31-bit sort keys of the embedding backward.
 */
rdcn_status rdcn_create(const rdcn_config* cfg, rdcn_handle** out);

/* Free the handle and its error word. NULL is accepted. */
rdcn_status rdcn_destroy(rdcn_handle* h);

/* Derived width d = F*D + Nd of x0 and of every x_l. */
rdcn_status rdcn_dim(const rdcn_handle* h, int64_t* d);

/*
 * Device bytes the caller must provide for a batch of `batch` samples:
 *   saved_bytes   -- activations written by rdcn_forward and read by rdcn_backward
 *   scratch_bytes -- temporary space for rdcn_forward / rdcn_backward
 * Both are 256-byte aligned sizes; the buffers must be 256-byte aligned.
 */
rdcn_status rdcn_workspace_bytes(const rdcn_handle* h, int64_t batch, size_t* saved_bytes, size_t* scratch_bytes);

/*
 * QR embedding gather (forward), section "Model Dictionary Compression":
 *   ids      : single-hot [batch, F] (offsets == NULL), or multi-hot CSR values
 *              with offsets [batch*F + 1] (int64) over bag index b*F + f;
 *              the offsets must be nondecreasing from offsets[0] >= 0 and ids
 *              must hold offsets[batch*F] values: the gather reads ids at those
 *              positions without a bound (it is not given their count)
 *   q_tables : [F, qr_rows_q, D],  r_tables : [F, m, D],  dense : [batch, Nd]
 *   x0       : [batch, d] output, all in the storage dtype.
 * Per element the combine is one float operation on the two table values
 * (product or sum), bags are pooled by float addition in bag order starting
 * from the first element (an empty bag gives +0), and the pooled float is
 * rounded to the storage type (bf16: round to nearest, ties to even). An id
 * outside [0, vocab) contributes nothing and raises the device error word
 * (see rdcn_check_device_errors).
 */
rdcn_status qr_embed_gather(rdcn_handle* h, int64_t batch, const void* ids, const int64_t* offsets,
                            const void* q_tables, const void* r_tables, const void* dense, void* x0,
                            void* stream);

/*
 * Middle-max 8-bit row-wise quantization of QR tables, section "Embedding
 * Table Quantization" (post-training, for serving). For each of the `rows`
 * rows of `tables` ([rows, emb_dim] in the storage dtype: all quotient tables
 * [F * qr_rows_q, D] or all remainder tables [F * m, D] of the handle's model)
 * with row minimum mn and maximum mx (a zero extreme counts as +0):
 *   middle = (mx * 128 + mn * 127) / 255,  scale = (mx - mn) / 255,
 *   code   = round((x - middle) / scale)   ties to even, in [-128, 127]
 * each a single IEEE float operation in that order; a constant row has scale 0
 * and codes 0. Outputs: codes [rows, D] int8 and params [rows, 2] float
 * (middle, scale). codes must be 8-byte aligned for bf16 models (4 for float),
 * params 8-byte aligned (RDCN_ERR_ARG otherwise); rows >= 2^32 gives
 * RDCN_ERR_UNSUPPORTED.
 */
rdcn_status qr_quantize_tables(rdcn_handle* h, int64_t rows, const void* tables, int8_t* codes, float* params,
                               void* stream);

/*
 * QR embedding gather from quantized tables (serving path): exactly
 * qr_embed_gather with every table value replaced by its dequantized value
 * middle + code * scale, computed with one rounding (fused multiply-add).
 * q_codes [F, qr_rows_q, D] and r_codes [F, m, D] int8, q_params / r_params
 * [F, rows, 2] float as written by qr_quantize_tables; ids, offsets, dense and
 * x0 as in qr_embed_gather. Alignment as for qr_quantize_tables.
 */
rdcn_status qr_embed_gather_q8(rdcn_handle* h, int64_t batch, const void* ids, const int64_t* offsets,
                               const int8_t* q_codes, const float* q_params, const int8_t* r_codes,
                               const float* r_params, const void* dense, void* x0, void* stream);

/*
 * Scratch bytes qr_embed_backward needs for `batch` samples holding `nnz` ids
 * in total (single-hot: nnz = batch * F). 0 for unhashed ids with tables of
 * at most 16384 rows (qr_rows_q and m), which take a one-kernel path.
 */
rdcn_status qr_embed_backward_workspace(const rdcn_handle* h, int64_t batch, int64_t nnz, size_t* scratch_bytes);

/*
 * QR embedding backward: table gradients from the x0 gradient, ACCUMULATED (+=)
 * into grad_q_tables [F, qr_rows_q, D] and grad_r_tables [F, m, D] (float).
 * This is the chain rule through the look-up and combine of section "Model
 * Dictionary Compression" (each id reads one quotient and one remainder row, so
 * its x0 gradient slice flows back to exactly those two rows). Besides the
 * arguments of qr_embed_gather it takes nnz (the id count, which sizes the sort
 * path) and the size of the caller's scratch, so that a too small workspace is an
 * error rather than an overrun.
 * grad_x0 is [batch, d] float (only its embedding columns are read). For every
 * valid id of bag (b, f) and g = grad_x0[b, f*D : (f+1)*D]:
 *   sum combine:     gQ_f[qi] += g,            gR_f[ri] += g
 *   product combine: gQ_f[qi] += g * R_f[ri],  gR_f[ri] += g * Q_f[qi]
 * No atomics: the order in which a row's contributions are added depends only
 * on the inputs and the configuration, so the result is deterministic.
 * ids/offsets/tables as in qr_embed_gather; nnz = number of ids (batch * F
 * when single-hot). scratch must hold qr_embed_backward_workspace() bytes (it
 * may be NULL when that is 0). grad_x0, grad_q_tables and
 * grad_r_tables must be 16-byte aligned (RDCN_ERR_ARG otherwise).
 */
rdcn_status qr_embed_backward(rdcn_handle* h, int64_t batch, int64_t nnz, const void* ids, const int64_t* offsets,
                              const void* q_tables, const void* r_tables, const float* grad_x0,
                              float* grad_q_tables, float* grad_r_tables, void* scratch, size_t scratch_bytes,
                              void* stream);

/*
 * qr_embed_backward without a caller-provided workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and errors as
 * qr_embed_backward, minus scratch: the sort path (hashed ids, or tables of more
 * than 16384 rows) uses a library-owned static device array of
 * RDCN_EMBED_STATIC_SCRATCH_BYTES per GPU, which the library holds from
 * rdcn_create until the process ends. RDCN_ERR_WORKSPACE (before any launch)
 * when qr_embed_backward_workspace() exceeds that size. The call allocates and
 * frees nothing. Every call on one GPU shares that GPU's array: calls that
 * overlap in time on one GPU (two streams, two host threads, two handles) race
 * and give wrong results; calls ordered on one stream are safe.
 */
#define RDCN_EMBED_STATIC_SCRATCH_BYTES (64ull << 20)
rdcn_status qr_embed_backward_static(rdcn_handle* h, int64_t batch, int64_t nnz, const void* ids,
                                     const int64_t* offsets, const void* q_tables, const void* r_tables,
                                     const float* grad_x0, float* grad_q_tables, float* grad_r_tables, void* stream);

/*
 * Residual-DCN forward, section "Residual DCN". x0 [batch, d] -> x_out = x_L
 * [batch, d], storage dtype. For each layer: [v; q; k] = W_l x_l (bf16 MFMA,
 * float accumulate); if alpha != 0, per sample S_ij = q_i k_j / tau, A = row
 * softmax of S, o = A v; h = beta v + alpha o; t = U_l h + b_l;
 * x_{l+1} = x0 * t + x_l. `saved` (saved_bytes) receives what rdcn_backward
 * needs and must stay untouched until then; `scratch` holds scratch_bytes (in
 * activation mode 2 the forward keeps one layer's f16 weight copies there; it
 * may be NULL in the other modes). With the attention term on, [v; q; k] are
 * kept in float (they feed the softmax, whose sharpness amplifies any rounding
 * of q and k); t is kept in the storage dtype and x_l and h as the activation
 * mode says (rdcn_act_mode). Deep stacks whose attention is close to one-hot
 * need mode 1 or 2 to keep gradients within a few percent of exact. In mode 2
 * the weights must be 16-byte aligned (RDCN_ERR_ARG otherwise).
 */
rdcn_status rdcn_forward(rdcn_handle* h, int64_t batch, const void* x0, const rdcn_weights* w, void* x_out,
                         void* saved, void* scratch, void* stream);

/*
 * Residual-DCN backward for the loss whose gradient w.r.t. x_L is grad_out
 * [batch, d] (storage dtype): the chain rule through the layer of section
 * "Residual DCN" (cross layer, attention between the two low-rank maps, skip
 * connection), which the paper states for the forward only. Writes
 * (overwrites) grad_x0 [batch, d] (float) and the float weight gradients in
 * `grads` (same shapes as the weights, summed over the batch). x0, w and saved
 * must be those of the matching rdcn_forward call.
 * The weight-gradient products (and the bias sums) may run on a second stream
 * that the handle owns (default priority; rdcn_set_side_stream can turn it off), forked from
 * `stream` after each layer's attention (layer 0, the last one, forks its bias
 * sums and gU after its pointwise kernel) and joined back to `stream` with events
 * before the call returns, on error returns too: work enqueued on `stream` after
 * the call sees every output, and capturing `stream` in a HIP graph captures both
 * streams. Two calls on one handle must not run concurrently on different streams.
 */
rdcn_status rdcn_backward(rdcn_handle* h, int64_t batch, const void* x0, const rdcn_weights* w, const void* saved,
                          const void* grad_out, float* grad_x0, const rdcn_weights* grads, void* scratch,
                          void* stream);

/*
 * Wait for `stream`, then read and clear the device error word:
 * RDCN_ERR_INDEX if any id outside [0, vocab) was met since the last check,
 * else RDCN_ERR_RANGE if an f16 activation or weight copy overflowed
 * (activation mode 2, the head's hidden layers),
 * RDCN_ERR_HIP on a runtime error, RDCN_OK otherwise.
 */
rdcn_status rdcn_check_device_errors(rdcn_handle* h, void* stream);

/*
 * Where rdcn_backward runs its bias sums and weight-gradient GEMMs (a scheduling
 * choice, not part of the paper's method): enable = 1 (the default) on the
 * handle's second stream beside the main chain, enable = 0 on `stream` itself,
 * so that every kernel runs alone and its measured time is its own (per-kernel
 * profiling). Results are bitwise the same either way. RDCN_ERR_ARG for a null
 * handle or another value.
 */
rdcn_status rdcn_set_side_stream(rdcn_handle* h, int32_t enable);

/* Static description of a status code. */
const char* rdcn_status_string(rdcn_status s);

/*
 * Kernel launch sites, for per-kernel timing. Each entry is one kernel,
 * except RDCN_KERNEL_EMB_SORT (all launches of one radix-sort pass sequence:
 * histogram, scan, scatter) and RDCN_KERNEL_EMB_REDUCE (segmented reduction
 * plus its fix-up).
 */
typedef enum rdcn_kernel {
    RDCN_KERNEL_GATHER = 0,         /* qr_embed_gather */
    RDCN_KERNEL_FWD_DOWN_GEMM = 1,  /* [v|q|k] = x_l W^T */
    RDCN_KERNEL_FWD_ATTENTION = 2,  /* per-sample softmax attention, h = beta v + alpha o */
    RDCN_KERNEL_FWD_UP_GEMM = 3,    /* t = h U^T + b, x_{l+1} = x0 * t + x_l */
    RDCN_KERNEL_BWD_POINTWISE = 4,  /* gt = g * x0, grad_x0 += g * t, bias partials */
    RDCN_KERNEL_BWD_BIAS = 5,       /* bias partials -> bias gradient */
    RDCN_KERNEL_BWD_GU_GEMM = 6,    /* gU = gt^T h */
    RDCN_KERNEL_BWD_GH_GEMM = 7,    /* gh = gt U */
    RDCN_KERNEL_BWD_ATTENTION = 8,  /* attention backward -> [gv|gq|gk] */
    RDCN_KERNEL_BWD_GW_GEMM = 9,    /* gW = [gv|gq|gk]^T x_l */
    RDCN_KERNEL_BWD_GX_GEMM = 10,   /* g_l = g_{l+1} + [gv|gq|gk] W */
    RDCN_KERNEL_SPLITK_REDUCE = 11, /* ordered sum of split-K partials of gU / gW */
    RDCN_KERNEL_EMB_KEYS = 12,      /* embedding backward: row keys */
    RDCN_KERNEL_EMB_SORT = 13,      /* embedding backward: stable radix sort */
    RDCN_KERNEL_EMB_REDUCE = 14,    /* embedding backward: segmented reduction + fix-up */
    RDCN_KERNEL_GATHER_Q8 = 15,     /* qr_embed_gather_q8 */
    RDCN_KERNEL_QUANTIZE = 16,      /* qr_quantize_tables */
    RDCN_KERNEL_HEAD_GATE = 17,     /* head: gate logits s_l = g_l . a_{l-1} + c_l */
    RDCN_KERNEL_HEAD_FWD_GEMM = 18, /* head: a_l = ReLU(a_{l-1} W_l^T + b_l) * sigmoid(s_l) */
    RDCN_KERNEL_HEAD_OUT = 19,      /* head: logit and isotonic calibration */
    RDCN_KERNEL_HEAD_LOSS = 20,     /* rdcn_head_logloss */
    RDCN_KERNEL_HEAD_OUT_BWD = 21,  /* head backward: calibration and logit gradients, top layer's G */
    RDCN_KERNEL_HEAD_GW_GEMM = 22,  /* head backward: gW_l = G_l^T a_{l-1} (plus split-K reduce) */
    RDCN_KERNEL_HEAD_GX_GEMM = 23,  /* head backward: G_{l-1} (or grad_x) from G_l W_l */
    RDCN_KERNEL_HEAD_GATE_BWD = 24, /* head backward: gate-logit gradients from the row partials */
    RDCN_KERNEL_HEAD_COLSUM = 25,   /* head backward: bias, gate and calibration gradients (column sums) */
    RDCN_KERNEL_EMB_FUSED = 26,     /* embedding backward in one kernel (per-slice sort + sums in LDS) */
    RDCN_KERNEL_COUNT = 27
} rdcn_kernel;

/*
 * ---------------------------------------------------------------------------
 * Head: the layers after the cross stack, for a Feed-style tower.
 *   - section "Dense Gating and Large MLP": wide ReLU layers on x = x_L, each
 *     hidden layer gated. Gate (a reading: the paper gives the idea, from
 *     GateNet, and its cost, negligible extra matrix work, not a formula): one
 *     scalar per sample and layer from the layer's own input,
 *       a_l = ReLU(W_l a_{l-1} + b_l) * sigmoid(g_l . a_{l-1} + c_l),  a_0 = x;
 *   - logit y = w_out . a_L + b_out;
 *   - section "Isotonic Calibration Layer", equation (calibration): with
 *     t = y - lo, bucket k = the largest j in [0, K-1] with t - step*j > 0 (0 if
 *     none; decided in float, each bound step*j rounded to float), v_i = step for
 *     i < k, v_k = t - step*k:
 *       y_cal = cal_b + sum_{i <= k} ReLU(e_i + cal_w_i) * v_i
 *     (below lo and above lo + K*step the first and last buckets extend
 *     linearly); e [batch, K] float is the per-sample calibration embedding,
 *     made upstream. y_cal is monotone non-decreasing in y.
 * bf16 models only. Each hidden activation a_l is kept twice: in f16, which
 * the next layer (an f16 MFMA product against an f16 copy of W_{l+1} made in
 * `saved`), the gate logits, the logit and the column sums of the output and
 * gate weight gradients read, and in bf16, which the weight-gradient products
 * and the ReLU masks read (|a_l| and |W_l| < 65520, else RDCN_ERR_RANGE is
 * flagged; rdcn_check_device_errors). Gate logits, y and y_cal are float.
 * ---------------------------------------------------------------------------
 */
#define RDCN_HEAD_MAX_HIDDEN 8

typedef struct rdcn_head_config {
    int32_t num_hidden;                    /* hidden layers, 1 .. RDCN_HEAD_MAX_HIDDEN */
    int32_t hidden[RDCN_HEAD_MAX_HIDDEN];  /* widths n_1 .. n_L, multiples of 8 (a width that is
                                              not one is run exactly by zero rows of padding) */
    int32_t gated;                         /* 0 or 1 */
    int32_t num_buckets;                   /* K, 1 .. 65536 */
    float bucket_lo;                       /* lo, finite */
    float bucket_step;                     /* step > 0, finite */
} rdcn_head_config;

/*
 * Head weights (entries at index >= num_hidden are ignored). n_0 = d.
 *   w[l]      : [n_l, n_{l-1}]  bf16       b[l]      : [n_l]  bf16
 *   gate_w[l] : [n_{l-1}]       bf16       gate_b[l] : [1]    bf16   (gated only)
 *   w_out     : [n_L] bf16,  b_out : [1] bf16
 *   cal_w     : [K] float,   cal_b : [1] float
 * Vector operands (w, b, gate_w, w_out) must be 16-byte aligned. Gradients use
 * the same struct with float buffers of the same shapes (overwritten).
 */
typedef struct rdcn_head_weights {
    void* w[RDCN_HEAD_MAX_HIDDEN];
    void* b[RDCN_HEAD_MAX_HIDDEN];
    void* gate_w[RDCN_HEAD_MAX_HIDDEN];
    void* gate_b[RDCN_HEAD_MAX_HIDDEN];
    void* w_out;
    void* b_out;
    void* cal_w;
    void* cal_b;
} rdcn_head_weights;

/*
 * Attach a head to the handle (replacing any earlier one); its input width is
 * the handle's d. RDCN_ERR_ARG for values out of range, RDCN_ERR_UNSUPPORTED
 * for a float model or a batch_max above 4194240.
 */
rdcn_status rdcn_head_configure(rdcn_handle* h, const rdcn_head_config* cfg);

/* Saved and scratch bytes of the head for `batch` samples (256-byte aligned buffers). */
rdcn_status rdcn_head_workspace_bytes(const rdcn_handle* h, int64_t batch, size_t* saved_bytes,
                                      size_t* scratch_bytes);

/*
 * Head forward: x [batch, d] bf16 (16-byte aligned; normally x_L of
 * rdcn_forward), e_cal [batch, K] float -> y_logit [batch] and y_cal [batch]
 * float. `saved` (rdcn_head_workspace_bytes) keeps the activations, gate logits
 * and logits for rdcn_head_backward.
 */
rdcn_status rdcn_head_forward(rdcn_handle* h, int64_t batch, const void* x, const float* e_cal,
                              const rdcn_head_weights* w, float* y_logit, float* y_cal, void* saved, void* stream);

/*
 * Log loss of a binary task on the calibrated logit z = y_cal, per sample:
 * loss = softplus(z) - label * z, grad = (sigmoid(z) - label) * scale (pass
 * scale = 1/batch for a mean loss). labels in [0, 1]; loss or grad may be NULL.
 */
rdcn_status rdcn_head_logloss(rdcn_handle* h, int64_t batch, const float* y_cal, const float* labels, float scale,
                              float* loss, float* grad, void* stream);

/*
 * Head backward for dLoss/dy_cal = grad_ycal [batch] float. Writes grad_x
 * [batch, d] bf16 (16-byte aligned; feeds rdcn_backward as grad_out), grad_e
 * [batch, K] float and every parameter gradient in `grads` (float, overwritten,
 * summed over the batch in a fixed order: deterministic). x, e_cal, w and saved
 * must be those of the matching rdcn_head_forward. ReLU'(0) = 0.
 */
rdcn_status rdcn_head_backward(rdcn_handle* h, int64_t batch, const void* x, const float* e_cal,
                               const rdcn_head_weights* w, const void* saved, const float* grad_ycal, void* grad_x,
                               float* grad_e, const rdcn_head_weights* grads, void* scratch, void* stream);

/*
 * Per-kernel timing with HIP events on the stream each kernel is launched on.
 * After rdcn_profile_start, each launch site whose bit (1 << rdcn_kernel) is
 * set in `kernel_mask` records an event before and after its kernel(s), up to
 * `max_launches` launches in total (events are created here, not during the
 * timed calls). rdcn_profile_stop waits for the
 * recorded events, writes the summed milliseconds and the number of timed
 * launches per rdcn_kernel into ms[RDCN_KERNEL_COUNT] and
 * launches[RDCN_KERNEL_COUNT], and turns timing off. Timing adds one event
 * pair per launch; it is meant for measurement runs.
 */
rdcn_status rdcn_profile_start(rdcn_handle* h, int32_t max_launches, uint32_t kernel_mask);
rdcn_status rdcn_profile_stop(rdcn_handle* h, double* ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* RDCN_H */
