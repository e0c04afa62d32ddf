/*
 * CPU oracle for the LiRank Residual-DCN + QR-embedding path -- TEST INFRASTRUCTURE.
 *
 * This file is the plain, slow, obviously-correct reference that the HIP path
 * is checked against. It is used only by the test-suite, the smoke check and
 * the CPU-baseline leg of the benchmark; the product library never links or
 * calls it, and it shares no code, header or table with the HIP sources.
 *
 * Paper: Borisyuk et al., "LiRank: Industrial Large Scale Ranking Models at
 * LinkedIn", KDD'24 (arXiv 2402.06859).
 *
 *   - QR index and combine: section "Model Dictionary Compression": an id is
 *     split into a quotient and a remainder by the remainder-table size m;
 *     each indexes its own small table and the two rows are aggregated by
 *     sum (the variant the paper found best) or elementwise product.
 *   - Embedding lookups replacing one-hot inputs, concatenated with dense
 *     features: section "Residual DCN" (first paragraph) and appendix "Feed
 *     Ranking Sparse ID features".
 *   - Cross layer: DCNv2 low-rank cross layer x_{l+1} = x0 * (U (V^T x_l) + b) + x_l
 *     (section "Residual DCN", first paragraph: the weight matrix replaced by
 *     two skinny matrices).
 *   - Attention low-rank cross net with skip connection and temperature:
 *     section "Residual DCN", second paragraph. The paper gives this only in
 *     prose (the defining figure is missing). Reading used here: the low-rank
 *     map is tripled into value/query/key maps; for one sample the r low-rank
 *     coordinates are r scalar tokens; S_ij = q_i k_j / tau; A = softmax over j;
 *     o = A v; the skip connection adds the value path: h = beta*v + alpha*o;
 *     then t = U h + b and x_{l+1} = x0 * t + x_l. With alpha = 0 this is the
 *     plain low-rank cross layer (scaled by beta).
 *
 * Precision: the cross stack runs in double from the storage values it is
 * given. The gather runs in float with the rounding the path defines: each
 * combined element is one float operation, bag pooling adds in bag order
 * starting from the first element (no +0.0 seed), and the pooled float is
 * rounded to bfloat16 (round to nearest, ties to even) when the storage type
 * is bfloat16. Build with -ffp-contract=off so that no multiply-add is fused.
 *
 * Every function returns the number of out-of-range ids it met (gather /
 * embedding backward) or 0, and -1 on bad arguments.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- QR index */

/* Rows of the quotient table that ids in [0, V) reach: ceil(V / m). */
int64_t orc_qr_quotient_rows(int64_t vocab, int64_t m) {
    if (vocab <= 0 || m <= 0) return -1;
    return (vocab + m - 1) / m;
}

/* id -> (quotient, remainder) = (floor(id / m), id mod m); ids outside [0, V)
 * get (-1, -1) and are counted. */
int64_t orc_qr_index(const int64_t* ids, int64_t n, int64_t vocab, int64_t m,
                     int64_t* qi, int64_t* ri) {
    if (m <= 0 || vocab <= 0) return -1;
    int64_t bad = 0;
    for (int64_t i = 0; i < n; ++i) {
        int64_t id = ids[i];
        if (id < 0 || id >= vocab) {
            qi[i] = -1;
            ri[i] = -1;
            ++bad;
            continue;
        }
        qi[i] = id / m;
        ri[i] = id - (id / m) * m;
    }
    return bad;
}

/* ------------------------------------------------------- bfloat16 rounding */

/* float -> nearest bfloat16 value (ties to even), returned as a float.
 * NaN stays a (quiet) NaN; overflow rounds to infinity. */
float orc_round_bf16(float x) {
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if ((u & 0x7fffffffu) > 0x7f800000u) {
        u = (u | 0x00400000u) & 0xffff0000u;
    } else {
        uint32_t keep_lsb = (u >> 16) & 1u;
        u = (u + 0x7fffu + keep_lsb) & 0xffff0000u;
    }
    float y;
    memcpy(&y, &u, sizeof y);
    return y;
}

void orc_round_bf16_array(const float* x, float* y, int64_t n) {
    for (int64_t i = 0; i < n; ++i) y[i] = orc_round_bf16(x[i]);
}

/* ------------------------------------------------------------------ gather */

enum { ORC_COMBINE_MUL = 0, ORC_COMBINE_SUM = 1 };

/*
 * x0[b, f*D + c] = round( pool_p  Q_f[qi_p, c] (op) R_f[ri_p, c] ),  x0[b, F*D + j] = dense[b, j]
 *
 * ids: single-hot [B, F] (offsets == NULL) or CSR values with offsets[B*F + 1]
 * over bag index b*F + f. q_tables [F, rows_q, D], r_tables [F, m, D], dense [B, Nd]:
 * storage values as float. An out-of-range id is counted and contributes
 * nothing to its bag; an empty bag gives +0.
 */
int64_t orc_gather(int64_t B, int64_t F, int64_t D, int64_t Nd, int64_t vocab, int64_t rows_q, int64_t m,
                   int combine, int round_bf16, const int64_t* ids, const int64_t* offsets,
                   const float* q_tables, const float* r_tables, const float* dense, float* x0) {
    if (B < 0 || F < 0 || D <= 0 || Nd < 0 || m <= 0) return -1;
    const int64_t d = F * D + Nd;
    int64_t bad = 0;
    float* acc = (float*)malloc(sizeof(float) * (size_t)D);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t f = 0; f < F; ++f) {
            int64_t begin, end;
            if (offsets) {
                begin = offsets[b * F + f];
                end = offsets[b * F + f + 1];
            } else {
                begin = b * F + f;
                end = begin + 1;
            }
            int started = 0;
            for (int64_t p = begin; p < end; ++p) {
                int64_t id = ids[p];
                if (id < 0 || id >= vocab) {
                    ++bad;
                    continue;
                }
                int64_t q = id / m;
                int64_t r = id - q * m;
                if (q >= rows_q) {
                    ++bad;
                    continue;
                }
                const float* qrow = q_tables + (f * rows_q + q) * D;
                const float* rrow = r_tables + (f * m + r) * D;
                for (int64_t c = 0; c < D; ++c) {
                    float e = (combine == ORC_COMBINE_MUL) ? qrow[c] * rrow[c] : qrow[c] + rrow[c];
                    acc[c] = started ? acc[c] + e : e;
                }
                started = 1;
            }
            float* dst = x0 + b * d + f * D;
            for (int64_t c = 0; c < D; ++c) {
                float v = started ? acc[c] : 0.0f;
                dst[c] = round_bf16 ? orc_round_bf16(v) : v;
            }
        }
        for (int64_t j = 0; j < Nd; ++j) x0[b * d + F * D + j] = dense[b * Nd + j];
    }
    free(acc);
    return bad;
}

/* --------------------------------------------------------------- attention */

/*
 * One sample's attention over its r low-rank coordinates (scalar tokens):
 *   S_ij = q_i k_j / tau,  A_ij = exp(S_ij - max_j S_ij) / sum_j exp(S_ij - max_j S_ij),
 *   o_i = sum_j A_ij v_j,  h_i = beta v_i + alpha o_i.
 * A (r*r, row-major) and o may be NULL. The row maximum is found by brute force.
 */
void orc_attention(int64_t r, double alpha, double beta, double tau, const double* q, const double* k,
                   const double* v, double* A, double* o, double* h) {
    double* row = (double*)malloc(sizeof(double) * (size_t)r);
    for (int64_t i = 0; i < r; ++i) {
        double mx = -INFINITY;
        for (int64_t j = 0; j < r; ++j) {
            row[j] = q[i] * k[j] / tau;
            if (row[j] > mx) mx = row[j];
        }
        double z = 0.0;
        for (int64_t j = 0; j < r; ++j) {
            row[j] = exp(row[j] - mx);
            z += row[j];
        }
        double oi = 0.0;
        for (int64_t j = 0; j < r; ++j) {
            row[j] /= z;
            oi += row[j] * v[j];
            if (A) A[i * r + j] = row[j];
        }
        if (o) o[i] = oi;
        h[i] = beta * v[i] + alpha * oi;
    }
    free(row);
}

/* ------------------------------------------------------------ cross stack */

/* Per-layer intermediates of one sample, kept for the backward pass. */
typedef struct {
    double* x;  /* [L+1][d]  x_0 .. x_L */
    double* v;  /* [L][r]   value of the attention (or of the only branch) */
    double* q;  /* [L][r]   (attention only) */
    double* k;  /* [L][r] */
    double* A;  /* [L][r][r] */
    double* o;  /* [L][r] */
    double* h;  /* [L][hr]  input of the up projection (hr = 2r with parallel branches) */
    double* t;  /* [L][d] */
} orc_tape;

static int tape_alloc(orc_tape* tp, int64_t L, int64_t d, int64_t r, int attn) {
    memset(tp, 0, sizeof *tp);
    tp->x = (double*)calloc((size_t)((L + 1) * d), sizeof(double));
    tp->v = (double*)calloc((size_t)(L * r), sizeof(double));
    tp->h = (double*)calloc((size_t)(L * 2 * r), sizeof(double));
    tp->t = (double*)calloc((size_t)(L * d), sizeof(double));
    if (attn) {
        tp->q = (double*)calloc((size_t)(L * r), sizeof(double));
        tp->k = (double*)calloc((size_t)(L * r), sizeof(double));
        tp->o = (double*)calloc((size_t)(L * r), sizeof(double));
        tp->A = (double*)calloc((size_t)(L * r * r), sizeof(double));
    }
    return tp->x && tp->v && tp->h && tp->t && (!attn || (tp->q && tp->k && tp->o && tp->A));
}

static void tape_free(orc_tape* tp) {
    free(tp->x); free(tp->v); free(tp->q); free(tp->k);
    free(tp->A); free(tp->o); free(tp->h); free(tp->t);
}

/*
 * Forward pass of one sample through L layers. Weights per layer l:
 *   w_down + l*n*r*d : [n*r, d], rows 0..r-1 = V^T, r..2r-1 = Q^T, 2r..3r-1 = K^T (n = 3 when
 *                      alpha != 0, else n = 1 and only V^T is present)
 *   u + l*d*hr       : [d, hr]
 *   bias + l*d       : [d]
 * With parallel branches (par != 0, alpha != 0) a plain low-rank cross net and an
 * attention low-rank cross net with their own weights run side by side: n = 4,
 * rows 0..r-1 = V1^T (plain branch), then V2^T, Q^T, K^T (attention branch);
 * h = [V1^T x | beta v2 + alpha A v2] has hr = 2r entries and U = [U1 | U2].
 */
static void sample_forward(int64_t d, int64_t r, int64_t L, double alpha, double beta, double tau, int par,
                           const double* x0, const double* w_down, const double* u, const double* bias,
                           orc_tape* tp) {
    const int attn = alpha != 0.0;
    par = par && attn;
    const int64_t n = attn ? (par ? 4 : 3) : 1;
    const int64_t hr = par ? 2 * r : r;
    memcpy(tp->x, x0, sizeof(double) * (size_t)d);
    for (int64_t l = 0; l < L; ++l) {
        const double* W = w_down + l * n * r * d;
        const double* U = u + l * d * hr;
        const double* bl = bias + l * d;
        const double* xl = tp->x + l * d;
        double* v = tp->v + l * r;
        double* h = tp->h + l * hr;
        double* t = tp->t + l * d;
        double* xn = tp->x + (l + 1) * d;
        if (par) {  /* plain branch: h[0..r) = V1^T x_l */
            for (int64_t i = 0; i < r; ++i) {
                double s = 0.0;
                for (int64_t c = 0; c < d; ++c) s += W[i * d + c] * xl[c];
                h[i] = s;
            }
        }
        const double* Wa = par ? W + r * d : W;  /* value, query, key rows of the attention branch */
        double* ha = par ? h + r : h;
        for (int64_t i = 0; i < r; ++i) {
            double s = 0.0;
            for (int64_t c = 0; c < d; ++c) s += Wa[i * d + c] * xl[c];
            v[i] = s;
        }
        if (attn) {
            double* q = tp->q + l * r;
            double* k = tp->k + l * r;
            for (int64_t i = 0; i < r; ++i) {
                double sq = 0.0, sk = 0.0;
                for (int64_t c = 0; c < d; ++c) {
                    sq += Wa[(r + i) * d + c] * xl[c];
                    sk += Wa[(2 * r + i) * d + c] * xl[c];
                }
                q[i] = sq;
                k[i] = sk;
            }
            orc_attention(r, alpha, beta, tau, q, k, v, tp->A + l * r * r, tp->o + l * r, ha);
        } else {
            for (int64_t i = 0; i < r; ++i) h[i] = beta * v[i];
        }
        for (int64_t c = 0; c < d; ++c) {
            double s = bl[c];
            for (int64_t i = 0; i < hr; ++i) s += U[c * hr + i] * h[i];
            t[c] = s;
            xn[c] = x0[c] * s + xl[c];
        }
    }
}

/* x_out[b] = x_L of sample b. x0 [B, d], x_out [B, d]. */
int orc_forward(int64_t B, int64_t d, int64_t r, int64_t L, double alpha, double beta, double tau, int par,
                const double* x0, const double* w_down, const double* u, const double* bias, double* x_out) {
    if (B < 0 || d <= 0 || r <= 0 || L <= 0 || tau <= 0.0) return -1;
    orc_tape tp;
    if (!tape_alloc(&tp, L, d, r, alpha != 0.0)) { tape_free(&tp); return -1; }
    for (int64_t b = 0; b < B; ++b) {
        sample_forward(d, r, L, alpha, beta, tau, par, x0 + b * d, w_down, u, bias, &tp);
        memcpy(x_out + b * d, tp.x + L * d, sizeof(double) * (size_t)d);
    }
    tape_free(&tp);
    return 0;
}

/*
 * Gradients of the scalar sum_b <grad_out[b], x_L[b]>:
 *   grad_x0 [B, d]            (overwritten)
 *   g_w_down [L, n*r, d], g_u [L, d, r], g_bias [L, d]  (overwritten, summed over the batch)
 * Chain rule per layer, last to first, with g = dLoss/dx_{l+1}:
 *   dt = g * x0;  gx0 += g * t;  g_bias += dt;  g_U += dt h^T;  dh = U^T dt
 *   attention: do = alpha dh;  dv = beta dh + A^T do;  dS_ij = A_ij do_i (v_j - o_i);
 *              dq_i = sum_j dS_ij k_j / tau;  dk_j = sum_i dS_ij q_i / tau
 *   plain:     dv = beta dh
 *   parallel branches: dh = [dh1 | dh2]; the plain branch's value gradient is dh1
 *              itself and the attention branch takes dh2 as above
 *   g_W += [dv; dq; dk] x_l^T;  g <- g + W^T [dv; dq; dk]   (with [dv1; dv2; dq; dk] in parallel)
 * and finally grad_x0 = gx0 + g (x0 is both the multiplier of every layer and the first input).
 * g_u is [L, d, hr].
 */
int orc_backward(int64_t B, int64_t d, int64_t r, int64_t L, double alpha, double beta, double tau, int par,
                 const double* x0, const double* w_down, const double* u, const double* bias,
                 const double* grad_out, double* grad_x0, double* g_w_down, double* g_u, double* g_bias) {
    if (B < 0 || d <= 0 || r <= 0 || L <= 0 || tau <= 0.0) return -1;
    const int attn = alpha != 0.0;
    par = par && attn;
    const int64_t n = attn ? (par ? 4 : 3) : 1;
    const int64_t hr = par ? 2 * r : r;
    memset(g_w_down, 0, sizeof(double) * (size_t)(L * n * r * d));
    memset(g_u, 0, sizeof(double) * (size_t)(L * d * hr));
    memset(g_bias, 0, sizeof(double) * (size_t)(L * d));
    orc_tape tp;
    double* g = (double*)malloc(sizeof(double) * (size_t)d);
    double* gn = (double*)malloc(sizeof(double) * (size_t)d);
    double* gx0 = (double*)malloc(sizeof(double) * (size_t)d);
    double* dt = (double*)malloc(sizeof(double) * (size_t)d);
    double* dh = (double*)malloc(sizeof(double) * (size_t)hr);
    double* dP = (double*)malloc(sizeof(double) * (size_t)(n * r));
    double* dS = (double*)malloc(sizeof(double) * (size_t)(r * r));
    int ok = tape_alloc(&tp, L, d, r, attn) && g && gn && gx0 && dt && dh && dP && dS;
    if (!ok) {
        tape_free(&tp); free(g); free(gn); free(gx0); free(dt); free(dh); free(dP); free(dS);
        return -1;
    }
    for (int64_t b = 0; b < B; ++b) {
        const double* xb0 = x0 + b * d;
        sample_forward(d, r, L, alpha, beta, tau, par, xb0, w_down, u, bias, &tp);
        memcpy(g, grad_out + b * d, sizeof(double) * (size_t)d);
        memset(gx0, 0, sizeof(double) * (size_t)d);
        for (int64_t l = L - 1; l >= 0; --l) {
            const double* W = w_down + l * n * r * d;
            const double* U = u + l * d * hr;
            const double* xl = tp.x + l * d;
            const double* h = tp.h + l * hr;
            const double* t = tp.t + l * d;
            double* gW = g_w_down + l * n * r * d;
            double* gU = g_u + l * d * hr;
            double* gb = g_bias + l * d;
            for (int64_t c = 0; c < d; ++c) {
                dt[c] = g[c] * xb0[c];
                gx0[c] += g[c] * t[c];
                gb[c] += dt[c];
                for (int64_t i = 0; i < hr; ++i) gU[c * hr + i] += dt[c] * h[i];
            }
            for (int64_t i = 0; i < hr; ++i) {
                double s = 0.0;
                for (int64_t c = 0; c < d; ++c) s += U[c * hr + i] * dt[c];
                dh[i] = s;
            }
            if (par)  /* plain branch: h1 = v1 */
                for (int64_t i = 0; i < r; ++i) dP[i] = dh[i];
            if (attn) {
                const double* dha = par ? dh + r : dh;
                double* dPa = par ? dP + r : dP;
                const double* A = tp.A + l * r * r;
                const double* v = tp.v + l * r;
                const double* q = tp.q + l * r;
                const double* k = tp.k + l * r;
                const double* o = tp.o + l * r;
                double* dv = dPa;
                double* dq = dPa + r;
                double* dk = dPa + 2 * r;
                for (int64_t j = 0; j < r; ++j) {
                    double s = 0.0;
                    for (int64_t i = 0; i < r; ++i) s += A[i * r + j] * alpha * dha[i];
                    dv[j] = beta * dha[j] + s;
                }
                for (int64_t i = 0; i < r; ++i)
                    for (int64_t j = 0; j < r; ++j) dS[i * r + j] = A[i * r + j] * alpha * dha[i] * (v[j] - o[i]);
                for (int64_t i = 0; i < r; ++i) {
                    double s = 0.0;
                    for (int64_t j = 0; j < r; ++j) s += dS[i * r + j] * k[j];
                    dq[i] = s / tau;
                }
                for (int64_t j = 0; j < r; ++j) {
                    double s = 0.0;
                    for (int64_t i = 0; i < r; ++i) s += dS[i * r + j] * q[i];
                    dk[j] = s / tau;
                }
            } else {
                for (int64_t i = 0; i < r; ++i) dP[i] = beta * dh[i];
            }
            for (int64_t i = 0; i < n * r; ++i)
                for (int64_t c = 0; c < d; ++c) gW[i * d + c] += dP[i] * xl[c];
            for (int64_t c = 0; c < d; ++c) {
                double s = g[c];
                for (int64_t i = 0; i < n * r; ++i) s += W[i * d + c] * dP[i];
                gn[c] = s;
            }
            memcpy(g, gn, sizeof(double) * (size_t)d);
        }
        for (int64_t c = 0; c < d; ++c) grad_x0[b * d + c] = gx0[c] + g[c];
    }
    tape_free(&tp);
    free(g); free(gn); free(gx0); free(dt); free(dh); free(dP); free(dS);
    return 0;
}

/* ------------------------------------------------------ embedding backward */

/*
 * Table gradients from the x0 gradient (accumulated with +=), in (b, p) order:
 * for every valid id of bag (b, f) with (qi, ri), and g = grad_x0[b, f*D : (f+1)*D]:
 *   sum combine:      gQ_f[qi] += g,            gR_f[ri] += g
 *   product combine:  gQ_f[qi] += g * R_f[ri],  gR_f[ri] += g * Q_f[qi]
 * (sum pooling gives every id of a bag the bag's gradient). grad_x0 [B, d] with
 * d = F*D + Nd; grad_q [F, rows_q, D], grad_r [F, m, D].
 */
int64_t orc_embed_backward(int64_t B, int64_t F, int64_t D, int64_t Nd, int64_t vocab, int64_t rows_q, int64_t m,
                           int combine, const int64_t* ids, const int64_t* offsets, const float* q_tables,
                           const float* r_tables, const double* grad_x0, double* grad_q, double* grad_r) {
    if (B < 0 || F < 0 || D <= 0 || Nd < 0 || m <= 0) return -1;
    const int64_t d = F * D + Nd;
    int64_t bad = 0;
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t f = 0; f < F; ++f) {
            int64_t begin = offsets ? offsets[b * F + f] : b * F + f;
            int64_t end = offsets ? offsets[b * F + f + 1] : begin + 1;
            const double* g = grad_x0 + b * d + f * D;
            for (int64_t p = begin; p < end; ++p) {
                int64_t id = ids[p];
                if (id < 0 || id >= vocab) { ++bad; continue; }
                int64_t q = id / m;
                int64_t r = id - q * m;
                if (q >= rows_q) { ++bad; continue; }
                double* gq = grad_q + (f * rows_q + q) * D;
                double* gr = grad_r + (f * m + r) * D;
                const float* qrow = q_tables + (f * rows_q + q) * D;
                const float* rrow = r_tables + (f * m + r) * D;
                for (int64_t c = 0; c < D; ++c) {
                    if (combine == ORC_COMBINE_MUL) {
                        gq[c] += g[c] * (double)rrow[c];
                        gr[c] += g[c] * (double)qrow[c];
                    } else {
                        gq[c] += g[c];
                        gr[c] += g[c];
                    }
                }
            }
        }
    }
    return bad;
}

/* ------------------------------------------- middle-max 8-bit table quantization */

/*
 * Section "Embedding Table Quantization": post-training row-wise quantization
 * of an embedding table X with bits = 8. For row i with minimum mn and
 * maximum mx:
 *   middle = (mx * 2^(bits-1) + mn * (2^(bits-1) - 1)) / (2^bits - 1)
 *   scale  = (mx - mn) / (2^bits - 1)
 *   code   = round((x - middle) / scale)          (lands in [-128, 127])
 *   value  = middle + code * scale                (dequantization)
 * In float, one rounding per operation in the order written: middle =
 * (mx*128 + mn*127) / 255, scale = (mx - mn) / 255, code = rint((x - middle) /
 * scale) with ties to even, clamped to [-128, 127]; an extreme that is a zero is
 * taken as +0 (the paper is silent on signed zeros). A constant row (mx == mn)
 * has scale 0 and all codes 0. Dequantization is middle + code*scale with a
 * single rounding (fused multiply-add).
 *
 * x [rows, D] (storage values as float) -> codes [rows, D], params [rows, 2] =
 * (middle, scale).
 */
int orc_quantize_rows(int64_t rows, int64_t D, const float* x, int8_t* codes, float* params) {
    if (rows < 0 || D <= 0) return -1;
    for (int64_t i = 0; i < rows; ++i) {
        const float* row = x + i * D;
        float mn = row[0], mx = row[0];
        for (int64_t c = 1; c < D; ++c) {
            if (row[c] < mn) mn = row[c];
            if (row[c] > mx) mx = row[c];
        }
        mn += 0.0f;  /* a zero extreme counts as +0 whichever zero was met first */
        mx += 0.0f;
        const float middle = (mx * 128.0f + mn * 127.0f) / 255.0f;
        const float scale = (mx - mn) / 255.0f;
        params[2 * i] = middle;
        params[2 * i + 1] = scale;
        for (int64_t c = 0; c < D; ++c) {
            float q = 0.0f;
            if (scale > 0.0f) {
                q = rintf((row[c] - middle) / scale);
                if (q < -128.0f) q = -128.0f;
                if (q > 127.0f) q = 127.0f;
            }
            codes[i * D + c] = (int8_t)q;
        }
    }
    return 0;
}

/* Dequantized table: value[i, c] = fma(code[i, c], scale_i, middle_i). */
int orc_dequantize_rows(int64_t rows, int64_t D, const int8_t* codes, const float* params, float* x) {
    if (rows < 0 || D <= 0) return -1;
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t c = 0; c < D; ++c) x[i * D + c] = fmaf((float)codes[i * D + c], params[2 * i + 1], params[2 * i]);
    return 0;
}

/*
 * Serving gather from quantized tables: exactly orc_gather with every table
 * value replaced by its dequantized value (the combine, pooling and rounding
 * are those of the gather).
 */
int64_t orc_gather_q8(int64_t B, int64_t F, int64_t D, int64_t Nd, int64_t vocab, int64_t rows_q, int64_t m,
                      int combine, int round_bf16, const int64_t* ids, const int64_t* offsets,
                      const int8_t* q_codes, const float* q_params, const int8_t* r_codes, const float* r_params,
                      const float* dense, float* x0) {
    if (B < 0 || F < 0 || D <= 0 || Nd < 0 || m <= 0 || rows_q <= 0) return -1;
    float* qt = (float*)malloc(sizeof(float) * (size_t)(F * rows_q * D + 1));
    float* rt = (float*)malloc(sizeof(float) * (size_t)(F * m * D + 1));
    orc_dequantize_rows(F * rows_q, D, q_codes, q_params, qt);
    orc_dequantize_rows(F * m, D, r_codes, r_params, rt);
    int64_t bad = orc_gather(B, F, D, Nd, vocab, rows_q, m, combine, round_bf16, ids, offsets, qt, rt, dense, x0);
    free(qt);
    free(rt);
    return bad;
}

/* ------------------------------------------------------- hashed front-end */

/*
 * Appendix "Vocabulary Compression" and section "Model Dictionary Compression":
 * a raw id is mapped by a stateless collision-resistant hash (Murmur) to int64,
 * the 64 bits are reinterpreted as two 32-bit numbers B (low half) and C (high
 * half), and each indexes its own set of QR tables. The hash here is
 * MurmurHash64A (the 64-bit member of Austin Appleby's MurmurHash2 family),
 * written from its published description: 8-byte little-endian blocks mixed by
 * multiply / xor-shift with m = 0xc6a4a7935bd1e995 and r = 47, a tail of up to 7
 * bytes folded in, then a final xor-shift / multiply / xor-shift.
 */
uint64_t orc_murmur64a(const void* key, int64_t len, uint64_t seed) {
    const uint64_t m = 0xc6a4a7935bd1e995ull;
    const int r = 47;
    const uint8_t* p = (const uint8_t*)key;
    uint64_t h = seed ^ ((uint64_t)len * m);
    const int64_t nblocks = len / 8;
    for (int64_t i = 0; i < nblocks; ++i) {
        uint64_t k = 0;
        for (int b = 7; b >= 0; --b) k = (k << 8) | p[8 * i + b];
        k *= m;
        k ^= k >> r;
        k *= m;
        h ^= k;
        h *= m;
    }
    const uint8_t* t = p + 8 * nblocks;
    const int rest = (int)(len & 7);
    if (rest > 0) {
        for (int b = rest - 1; b >= 0; --b) h ^= (uint64_t)t[b] << (8 * b);
        h *= m;
    }
    h ^= h >> r;
    h *= m;
    h ^= h >> r;
    return h;
}

/* Hash of every id: its 8 bytes in little-endian order. */
void orc_hash_ids(const int64_t* ids, int64_t n, uint64_t seed, uint64_t* out) {
    for (int64_t i = 0; i < n; ++i) {
        uint8_t bytes[8];
        uint64_t v = (uint64_t)ids[i];
        for (int b = 0; b < 8; ++b) bytes[b] = (uint8_t)(v >> (8 * b));
        out[i] = orc_murmur64a(bytes, 8, seed);
    }
}

/*
 * Gather with the hashed front-end. q_tables [F, 2, rows_q, D] and r_tables
 * [F, 2, m, D]: pair 0 serves the low half B, pair 1 the high half C of each
 * id's hash; each half x in [0, 2^32) is QR-split (qi = x / m, ri = x mod m; needs
 * rows_q * m >= 2^32). The element of one id is (Q0[qi_B] op R0[ri_B]) + (Q1[qi_C]
 * op R1[ri_C]) in float: each combine one float operation, the two halves summed
 * (the paper does not say how the two look-ups are aggregated; the sum is the
 * aggregation it found best for QR). Bags pool as in orc_gather. Every id is valid.
 */
int64_t orc_gather_hashed(int64_t B, int64_t F, int64_t D, int64_t Nd, int64_t rows_q, int64_t m, int combine,
                          int round_bf16, uint64_t seed, const int64_t* ids, const int64_t* offsets,
                          const float* q_tables, const float* r_tables, const float* dense, float* x0) {
    if (B < 0 || F < 0 || D <= 0 || Nd < 0 || m <= 0 || rows_q <= 0) return -1;
    if ((uint64_t)rows_q * (uint64_t)m < ((uint64_t)1 << 32)) return -1;
    const int64_t d = F * D + Nd;
    float* acc = (float*)malloc(sizeof(float) * (size_t)D);
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t f = 0; f < F; ++f) {
            int64_t begin = offsets ? offsets[b * F + f] : b * F + f;
            int64_t end = offsets ? offsets[b * F + f + 1] : begin + 1;
            int started = 0;
            for (int64_t p = begin; p < end; ++p) {
                uint64_t hsh;
                orc_hash_ids(&ids[p], 1, seed, &hsh);
                const uint64_t half[2] = {hsh & 0xffffffffull, hsh >> 32};
                const float* qrow[2];
                const float* rrow[2];
                for (int s = 0; s < 2; ++s) {
                    const uint64_t qi = half[s] / (uint64_t)m, ri = half[s] % (uint64_t)m;
                    qrow[s] = q_tables + ((f * 2 + s) * rows_q + (int64_t)qi) * D;
                    rrow[s] = r_tables + ((f * 2 + s) * m + (int64_t)ri) * D;
                }
                for (int64_t c = 0; c < D; ++c) {
                    float e0 = (combine == ORC_COMBINE_MUL) ? qrow[0][c] * rrow[0][c] : qrow[0][c] + rrow[0][c];
                    float e1 = (combine == ORC_COMBINE_MUL) ? qrow[1][c] * rrow[1][c] : qrow[1][c] + rrow[1][c];
                    float e = e0 + e1;
                    acc[c] = started ? acc[c] + e : e;
                }
                started = 1;
            }
            float* dst = x0 + b * d + f * D;
            for (int64_t c = 0; c < D; ++c) {
                float v = started ? acc[c] : 0.0f;
                dst[c] = round_bf16 ? orc_round_bf16(v) : v;
            }
        }
        for (int64_t j = 0; j < Nd; ++j) x0[b * d + F * D + j] = dense[b * Nd + j];
    }
    free(acc);
    return 0;
}

/*
 * Table gradients of the hashed gather (accumulated, in (b, p) order), g =
 * grad_x0[b, f*D : (f+1)*D], for both halves s of every id:
 *   sum combine:      gQs[qi_s] += g,               gRs[ri_s] += g
 *   product combine:  gQs[qi_s] += g * Rs[ri_s],    gRs[ri_s] += g * Qs[qi_s]
 * grad_q [F, 2, rows_q, D], grad_r [F, 2, m, D].
 */
int64_t orc_embed_backward_hashed(int64_t B, int64_t F, int64_t D, int64_t Nd, int64_t rows_q, int64_t m,
                                  int combine, uint64_t seed, const int64_t* ids, const int64_t* offsets,
                                  const float* q_tables, const float* r_tables, const double* grad_x0,
                                  double* grad_q, double* grad_r) {
    if (B < 0 || F < 0 || D <= 0 || Nd < 0 || m <= 0 || rows_q <= 0) return -1;
    if ((uint64_t)rows_q * (uint64_t)m < ((uint64_t)1 << 32)) return -1;
    const int64_t d = F * D + Nd;
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t f = 0; f < F; ++f) {
            int64_t begin = offsets ? offsets[b * F + f] : b * F + f;
            int64_t end = offsets ? offsets[b * F + f + 1] : begin + 1;
            const double* g = grad_x0 + b * d + f * D;
            for (int64_t p = begin; p < end; ++p) {
                uint64_t hsh;
                orc_hash_ids(&ids[p], 1, seed, &hsh);
                for (int s = 0; s < 2; ++s) {
                    const uint64_t x = s ? hsh >> 32 : hsh & 0xffffffffull;
                    const int64_t qi = (int64_t)(x / (uint64_t)m), ri = (int64_t)(x % (uint64_t)m);
                    double* gq = grad_q + ((f * 2 + s) * rows_q + qi) * D;
                    double* gr = grad_r + ((f * 2 + s) * m + ri) * D;
                    const float* qrow = q_tables + ((f * 2 + s) * rows_q + qi) * D;
                    const float* rrow = r_tables + ((f * 2 + s) * m + ri) * D;
                    for (int64_t c = 0; c < D; ++c) {
                        if (combine == ORC_COMBINE_MUL) {
                            gq[c] += g[c] * (double)rrow[c];
                            gr[c] += g[c] * (double)qrow[c];
                        } else {
                            gq[c] += g[c];
                            gr[c] += g[c];
                        }
                    }
                }
            }
        }
    }
    return 0;
}
