/*
 * Oracle for the routed MoE FFN forward of EPS-MoE (arXiv 2410.12247).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously correct
 * CPU statement of what the GPU path computes.  Only the tests, the smoke
 * check and the CPU-baseline leg of the benchmark may load it.  It shares
 * no code, header, table or helper with the HIP library, and it includes
 * nothing from it.
 *
 * What it computes, step by step, for one GPU's share of experts
 * [e0, e0 + EL) of E router experts, T tokens of width H, SwiGLU width I:
 *
 *   1. Router logits (the "topKGating" operator named among the memory-bound
 *      MoE operators in Sec. 3.3): z[t][e] = sum_h x[t][h] * Wr[e][h], one
 *      fp32 fused multiply-add per h in ascending h starting from +0, then
 *      one fp32 add of bias[e] when a bias is given.  The paper fixes
 *      neither precision nor order; fp32 with this order is the reading
 *      used (the GPU reaches the same bits).
 *   2. Top-k (Sec. 3.2 defines k as the number of experts a token selects out
 *      of E): the k largest fp32 logits, ordered by (logit descending,
 *      expert index ascending); -0 and +0 compare equal.
 *   3. Routing weights: softmax in fp64, rounded to fp32 once.  With
 *      renormalisation the softmax runs over the k selected logits; without
 *      it, over all E logits.
 *   4. Dispatch (Fig. 7a caption: each expert takes its tokens in ascending
 *      token order; Sec. 4.3: weights split by expert, inputs split by rows):
 *      rows ordered by (local expert ascending, token ascending).  counts,
 *      offsets (exclusive prefix of counts), sorted_slot (row -> t*k+j) and
 *      slot_row (slot -> row, -1 for a slot whose expert is not local).
 *   5. Expert FFN (the Gate, Up and Down GEMMs of the one-layer ablation in
 *      Sec. 5.2 with the silu activation of Sec. 3.3): per row,
 *      g = Wg_e x, u = Wu_e x, a = silu(g) * u, y = Wd_e a, all in fp64 from
 *      the bf16 inputs, rounded to fp32 once at the end.
 *   6. Combine (LocalReduce, Fig. 7b caption): y[t] = sum over slots j whose
 *      expert is local of w[t][j] * y_row, in fp64 with the fp32 weights of
 *      step 3 and the fp32 expert rows of step 5; plus the shared experts'
 *      output (a plain SwiGLU FFN on every token, fp64) when present;
 *      rounded to fp32 once.
 *
 * bf16 inputs arrive as raw 16-bit patterns and are widened exactly
 * (bits << 16).  Every parallel loop computes each output from its own
 * inputs only, so results do not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static float bf16_to_f32(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* ---- step 1: router logits --------------------------------------------- */
void oracle_router_logits(const uint16_t *x, const float *wr, const float *bias,
                          int64_t T, int H, int E, float *z) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const uint16_t *xt = x + t * (int64_t)H;
        for (int e = 0; e < E; ++e) {
            const float *we = wr + (int64_t)e * H;
            float acc = 0.0f;
            for (int h = 0; h < H; ++h)
                acc = fmaf(bf16_to_f32(xt[h]), we[h], acc);
            if (bias) acc = acc + bias[e];
            z[t * E + e] = acc;
        }
    }
}

/* ---- steps 2-3: top-k selection and softmax weights --------------------- */
/* 1 when logit a of expert ea ranks ahead of logit b of expert eb. */
static int ranks_ahead(float a, int ea, float b, int eb) {
    if (a > b) return 1;
    if (a < b) return 0;
    return ea < eb; /* equal values (including -0 == +0): lower index first */
}

void oracle_topk(const float *z, int64_t T, int E, int k, int renorm,
                 int32_t *ids, float *w) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const float *zt = z + t * E;
        int32_t *it = ids + t * k;
        /* selection: k passes, each taking the best expert not yet taken */
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                int taken = 0;
                for (int q = 0; q < j; ++q)
                    if (it[q] == e) taken = 1;
                if (taken) continue;
                if (best < 0 || ranks_ahead(zt[e], e, zt[best], best)) best = e;
            }
            it[j] = best;
        }
        /* softmax in fp64 */
        double zmax = zt[it[0]];
        double denom = 0.0;
        if (renorm) {
            for (int j = 0; j < k; ++j) denom += exp((double)zt[it[j]] - zmax);
        } else {
            for (int e = 0; e < E; ++e) denom += exp((double)zt[e] - zmax);
        }
        for (int j = 0; j < k; ++j)
            w[t * k + j] = (float)(exp((double)zt[it[j]] - zmax) / denom);
    }
}

/* ---- step 4: dispatch order ---------------------------------------------- */
/* Returns R, the number of routed local rows. */
int64_t oracle_dispatch(const int32_t *ids, int64_t T, int k, int e0, int EL,
                        int32_t *counts, int32_t *offsets, int32_t *sorted_slot,
                        int32_t *slot_row) {
    for (int e = 0; e < EL; ++e) counts[e] = 0;
    for (int64_t s = 0; s < T * k; ++s) {
        int e = ids[s] - e0;
        if (e >= 0 && e < EL) counts[e] += 1;
    }
    offsets[0] = 0;
    for (int e = 0; e < EL; ++e) offsets[e + 1] = offsets[e] + counts[e];
    /* fill each expert's segment in ascending slot order; a token selects an
       expert at most once, so slot order within an expert is token order */
    int32_t *fill = (int32_t *)malloc(sizeof(int32_t) * (size_t)(EL > 0 ? EL : 1));
    for (int e = 0; e < EL; ++e) fill[e] = offsets[e];
    for (int64_t s = 0; s < T * k; ++s) {
        int e = ids[s] - e0;
        if (e >= 0 && e < EL) {
            int32_t r = fill[e]++;
            sorted_slot[r] = (int32_t)s;
            slot_row[s] = r;
        } else {
            slot_row[s] = -1;
        }
    }
    free(fill);
    return offsets[EL];
}

/* ---- step 5: one SwiGLU FFN row ------------------------------------------ */
/* y = Wd (silu(Wg x) * (Wu x)), fp64 throughout; wg, wu are [I][H],
 * wd is [H][ldd] (ldd >= I: the expert's down matrix may be a column block
 * of a wider one).  out_f64 receives H fp64 values. */
static void swiglu_row_f64(const uint16_t *xrow, const uint16_t *wg, const uint16_t *wu,
                           const uint16_t *wd, int H, int I, int64_t ldd,
                           double *a_scratch, double *out_f64) {
    for (int i = 0; i < I; ++i) {
        const uint16_t *gi = wg + (int64_t)i * H;
        const uint16_t *ui = wu + (int64_t)i * H;
        double g = 0.0, u = 0.0;
        for (int h = 0; h < H; ++h) {
            double xv = bf16_to_f32(xrow[h]);
            g += (double)bf16_to_f32(gi[h]) * xv;
            u += (double)bf16_to_f32(ui[h]) * xv;
        }
        double silu = g / (1.0 + exp(-g));
        a_scratch[i] = silu * u;
    }
    for (int h = 0; h < H; ++h) {
        const uint16_t *dh = wd + (int64_t)h * ldd;
        double acc = 0.0;
        for (int i = 0; i < I; ++i) acc += (double)bf16_to_f32(dh[i]) * a_scratch[i];
        out_f64[h] = acc;
    }
}

/* Expert FFN of one dispatched row of local expert el: x row xrow [H],
 * expert weight stacks wg, wu [EL][I][H] and wd [EL][H][I]; y_row [H] fp32. */
void oracle_expert_row(const uint16_t *xrow, const uint16_t *wg, const uint16_t *wu,
                       const uint16_t *wd, int H, int I, int el, float *y_row) {
    double *a = (double *)malloc(sizeof(double) * (size_t)I);
    double *o = (double *)malloc(sizeof(double) * (size_t)H);
    const int64_t wsz = (int64_t)I * H;
    swiglu_row_f64(xrow, wg + el * wsz, wu + el * wsz, wd + el * wsz, H, I, I, a, o);
    for (int h = 0; h < H; ++h) y_row[h] = (float)o[h];
    free(a);
    free(o);
}

/* All dispatched rows: y_perm[r] = FFN_{expert of r}(x[token of r]). */
void oracle_expert_rows(const uint16_t *x, const int32_t *sorted_slot, const int32_t *offsets,
                        const uint16_t *wg, const uint16_t *wu, const uint16_t *wd,
                        int H, int I, int k, int EL, float *y_perm) {
    for (int el = 0; el < EL; ++el) {
        int32_t rb = offsets[el], re = offsets[el + 1];
#pragma omp parallel for schedule(dynamic, 1)
        for (int32_t r = rb; r < re; ++r) {
            int64_t t = sorted_slot[r] / k;
            oracle_expert_row(x + t * H, wg, wu, wd, H, I, el, y_perm + (int64_t)r * H);
        }
    }
}

/* Selected rows: y_rows[n] = FFN of local expert el[n] applied to token
 * tok[n] (any list of pairs, e.g. a sample of dispatched rows). */
void oracle_expert_row_list(const uint16_t *x, const int64_t *tok, const int32_t *el,
                            int64_t n_rows, const uint16_t *wg, const uint16_t *wu,
                            const uint16_t *wd, int H, int I, float *y_rows) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t n = 0; n < n_rows; ++n)
        oracle_expert_row(x + tok[n] * H, wg, wu, wd, H, I, el[n], y_rows + n * H);
}

/* ---- steps 5-6 for a subset of tokens ------------------------------------ */
/* Output rows y_sel[n] = MoE FFN of token tok[n], given the routing of that
 * token (ids, w as produced by oracle_topk).  Shared experts: n_shared
 * SwiGLU FFNs of width Is each, weights wsg, wsu [n_shared*Is][H] and wsd
 * [H][n_shared*Is] (expert s owns gate/up rows and down columns
 * [s*Is, (s+1)*Is)); pass n_shared = 0 for none.  Each token's expert rows
 * are computed directly, without the dispatch order, so this path is
 * independent of step 4. */
void oracle_moe_tokens(const uint16_t *x, const int32_t *ids, const float *w,
                       const int64_t *tok, int64_t n_tok, int H, int I, int k,
                       int e0, int EL, const uint16_t *wg, const uint16_t *wu,
                       const uint16_t *wd, int n_shared, int Is, const uint16_t *wsg,
                       const uint16_t *wsu, const uint16_t *wsd, float *y_sel) {
    const int64_t wsz = (int64_t)I * H;
    int amax = I > Is ? I : Is;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t n = 0; n < n_tok; ++n) {
        int64_t t = tok[n];
        const uint16_t *xrow = x + t * H;
        double *a = (double *)malloc(sizeof(double) * (size_t)(amax > 0 ? amax : 1));
        double *o = (double *)malloc(sizeof(double) * (size_t)H);
        double *acc = (double *)calloc((size_t)H, sizeof(double));
        for (int j = 0; j < k; ++j) {
            int el = ids[t * k + j] - e0;
            if (el < 0 || el >= EL) continue;
            swiglu_row_f64(xrow, wg + el * wsz, wu + el * wsz, wd + el * wsz, H, I, I, a, o);
            double wj = w[t * k + j];
            /* the expert row is an fp32 value of the method (step 5) */
            for (int h = 0; h < H; ++h) acc[h] += wj * (double)(float)o[h];
        }
        for (int s = 0; s < n_shared; ++s) {
            const int64_t ldd = (int64_t)n_shared * Is;
            swiglu_row_f64(xrow, wsg + (int64_t)s * Is * H, wsu + (int64_t)s * Is * H,
                           wsd + (int64_t)s * Is, H, Is, ldd, a, o);
            for (int h = 0; h < H; ++h) acc[h] += o[h];
        }
        for (int h = 0; h < H; ++h) y_sel[n * H + h] = (float)acc[h];
        free(a);
        free(o);
        free(acc);
    }
}

/* ---- step 6 from dispatched rows ----------------------------------------- */
/* y[t] = sum_j w[t][j] * y_perm[slot_row[t*k+j]] (+ y_init[t] when given). */
void oracle_combine(const float *y_perm, const int32_t *slot_row, const float *w,
                    const float *y_init, int64_t T, int H, int k, float *y) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int h = 0; h < H; ++h) {
            double acc = y_init ? (double)y_init[t * H + h] : 0.0;
            for (int j = 0; j < k; ++j) {
                int32_t r = slot_row[t * k + j];
                if (r < 0) continue;
                acc += (double)w[t * k + j] * (double)y_perm[(int64_t)r * H + h];
            }
            y[t * H + h] = (float)acc;
        }
    }
}
