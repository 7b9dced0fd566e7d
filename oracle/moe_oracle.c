/*
 * moe_oracle.c -- CPU oracle for one MoE layer's forward (SAEM, arXiv 2608.21614).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the package smoke check and the bench's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with the
 * HIP library; the two meet only in the seeded input buffers.
 *
 * Plain loops, fp64 arithmetic.  Inputs are read exactly: fp32 elements, or
 * bf16 bit patterns widened to fp32 and then to double (both exact).
 *
 * What the layer computes, in the paper's order (Section IV-A overview,
 * Section IV-D.2 hybrid pipeline, Section IV-E.1 token repacking):
 *   1. router scores and top-k gating (Section II-A: a router picks the top-k
 *      experts of each token);
 *   2. expert-aligned token repacking: group the (token, expert) pairs by expert
 *      so that every expert's tokens are contiguous (Section IV-E.1 and its
 *      worked four-token example);
 *   3. partition of the repacked batch by the residency map into GPU-bound and
 *      host-bound groups (Section IV-D.2);
 *   4. every expert runs once over its dense buffer (Section IV-E.1);
 *   5. the per-expert outputs are merged back into token order (Section IV-D.2).
 * The paper does not spell out the gate or the expert MLP.  This oracle reads
 * them as: softmax over the k selected scores (renormalised top-k gate) and a
 * SwiGLU MLP y = (silu(x W1) * (x W3)) W2 without biases.
 *
 * Parallelism: OpenMP over independent outputs only; every output element is a
 * plain sequential sum, so results do not depend on the thread count.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1

/* Exact value of element i of a stored tensor. */
static double elem(const void* p, int64_t i, int dtype) {
    if (dtype == ORACLE_BF16) {
        uint32_t bits = ((uint32_t)((const uint16_t*)p)[i]) << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return (double)((const float*)p)[i];
}

int oracle_version(void) { return 1; }

/* Threads the OpenMP loops below use. */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Threads for the following calls; every loop splits outputs, never a sum, so the
 * results do not depend on it. */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/*
 * Router scores (Section II-A): score[t][e] = sum_h x[t][h] * w_router[e][h] + bias[e].
 * x is [T,H], w_router is [E,H] (row e scores expert e), bias is [E] fp32 or NULL.
 * The bias is part of the score: it moves both the selection and the gate.
 */
void oracle_router_logits(int64_t T, int64_t H, int64_t E, int dtype, const void* x,
                          const void* w_router, const float* bias, double* logits) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t e = 0; e < E; ++e) {
            double s = 0.0;
            for (int64_t h = 0; h < H; ++h)
                s += elem(x, t * H + h, dtype) * elem(w_router, e * H + h, dtype);
            if (bias) s += (double)bias[e];
            logits[t * E + e] = s;
        }
    }
}

/*
 * Top-k gating (Section II-A) on given scores.
 * idx[t][j]: the j-th selected expert, in order of decreasing score; equal
 * scores go to the lower expert index first.  -inf scores are allowed.
 * w[t][j] = exp(s_j - s_0) / sum_{j'} exp(s_j' - s_0): the softmax over the k
 * selected scores (equal to the full softmax renormalised over the selection).
 * A term whose score equals the top score counts as exactly 1, so a token whose
 * selected scores are all equal (including all -inf) gets w = 1/k.
 */
void oracle_topk(int64_t T, int64_t E, int64_t k, const double* logits, int32_t* idx, double* w) {
    for (int64_t t = 0; t < T; ++t) {
        const double* s = logits + t * E;
        unsigned char* taken = (unsigned char*)calloc((size_t)E, 1);
        for (int64_t j = 0; j < k; ++j) {
            int64_t best = -1;
            for (int64_t e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || s[e] > s[best]) best = e; /* strict: ties keep the lower index */
            }
            taken[best] = 1;
            idx[t * k + j] = (int32_t)best;
        }
        free(taken);
        double top = s[idx[t * k]];
        double z = 0.0;
        for (int64_t j = 0; j < k; ++j) {
            double sj = s[idx[t * k + j]];
            double term = (sj == top) ? 1.0 : exp(sj - top);
            w[t * k + j] = term;
            z += term;
        }
        for (int64_t j = 0; j < k; ++j) w[t * k + j] /= z;
    }
}

/*
 * Expert-aligned token repacking (Section IV-E.1) with the residency split of
 * Section IV-D.2.  Pair q = t*k + j is the j-th selected expert of token t.
 *   counts[e]    number of pairs routed to expert e;
 *   group order  resident experts by ascending id, then offloaded experts by
 *                ascending id;
 *   seg_start[e] first packed row of expert e (sum of the counts of the experts
 *                before it in group order);
 *   perm[p]      the pair stored at packed row p: each expert's pairs are
 *                contiguous, in ascending token order;
 *   inv_perm[q]  the packed row of pair q;
 *   n_res        number of pairs bound for resident experts: rows [0, n_res)
 *                are the GPU-bound group, rows [n_res, T*k) the host-bound one.
 * resident[e] is nonzero for a GPU-resident expert.
 * Returns 0, or -1 if idx holds an expert id outside [0, E).
 */
int oracle_repack(int64_t T, int64_t E, int64_t k, const int32_t* idx, const uint8_t* resident,
                  int32_t* counts, int32_t* seg_start, int32_t* perm, int32_t* inv_perm,
                  int32_t* n_res) {
    int64_t P = T * k;
    for (int64_t e = 0; e < E; ++e) counts[e] = 0;
    for (int64_t q = 0; q < P; ++q) {
        if (idx[q] < 0 || idx[q] >= E) return -1;
        counts[idx[q]] += 1;
    }
    int64_t row = 0, nres = 0;
    for (int pass = 0; pass < 2; ++pass) {          /* pass 0: resident, pass 1: offloaded */
        for (int64_t e = 0; e < E; ++e) {
            int is_res = resident[e] != 0;
            if ((pass == 0) != is_res) continue;
            seg_start[e] = (int32_t)row;
            for (int64_t t = 0; t < T; ++t)
                for (int64_t j = 0; j < k; ++j)
                    if (idx[t * k + j] == e) perm[row++] = (int32_t)(t * k + j);
            if (is_res) nres += counts[e];
        }
    }
    for (int64_t p = 0; p < P; ++p) inv_perm[perm[p]] = (int32_t)p;
    *n_res = (int32_t)nres;
    return 0;
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/*
 * One expert over its dense input buffer (Section IV-E.1: one batched execution
 * per expert).  Row r of the buffer is token row_token[r] of x ([*,H]).
 *   g = x W1, u = x W3, a = silu(g) * u, y = a W2, silu(z) = z / (1 + e^-z).
 * Storage: w13 is [2F,H], row f < F holds column f of W1 and row F+f column f
 * of W3; w2 is [H,F], row h holds column h of W2.  y is [n,H], fp64.
 */
void oracle_expert_ffn(int64_t n, int64_t H, int64_t F, int dtype, const void* x,
                       const int32_t* row_token, const void* w13, const void* w2, double* y) {
    double* a = (double*)malloc(sizeof(double) * (size_t)(F > 0 ? F : 1));
    for (int64_t r = 0; r < n; ++r) {
        int64_t t = row_token[r];
#pragma omp parallel for schedule(static)
        for (int64_t f = 0; f < F; ++f) {
            double g = 0.0, u = 0.0;
            for (int64_t h = 0; h < H; ++h) {
                double xv = elem(x, t * H + h, dtype);
                g += xv * elem(w13, f * H + h, dtype);
                u += xv * elem(w13, (F + f) * H + h, dtype);
            }
            a[f] = silu(g) * u;
        }
#pragma omp parallel for schedule(static)
        for (int64_t h = 0; h < H; ++h) {
            double s = 0.0;
            for (int64_t f = 0; f < F; ++f) s += a[f] * elem(w2, h * F + f, dtype);
            y[r * H + h] = s;
        }
    }
    free(a);
}
