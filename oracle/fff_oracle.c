/*
 * fff_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU reference for fast-feedforward (FFF) inference: the
 * conditional matrix multiplication (CMM) tree descent followed by the output
 * accumulation, from "Exponentially Faster Language Modeling" (Belcak and
 * Wattenhofer, 2023), Algorithm 1 with the model changes of Section 2.1.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * load this library; the product path never does, and it shares no code with
 * the HIP kernels.
 *
 * What is computed, for every token b and tree t (inputs widened exactly to
 * double; bf16 bit patterns become float, then double):
 *
 *   n = 0 (the root), and for levels l = 0 .. D:
 *     logit = sum_i x[b,i] * W_in[t,n,i]                  (CMM dot product)
 *     a     = act(logit)                                   (GELU at every node)
 *     y[b] += a * W_out[t,n,:]                             (every node has output weights)
 *     if l < D: n = 2n + 1 + (logit > 0)                   (child from the sign)
 *
 * and y sums over the trees (multiple trees, Section 2.1).
 *
 * Readings of the paper (its printed listing is off by one in places):
 *   - depth D counts edges: a tree has N = 2^(D+1) - 1 nodes in heap order
 *     and a token visits D+1 of them, one per level (Table 1's neuron counts,
 *     12 of 4095 at depth 11);
 *   - the logit is computed at every level including the root, and the
 *     activation of a node multiplies that same node's output row; the rows
 *     are summed into the token's output, not assigned to a column;
 *   - the comparison is strict: a logit of exactly 0 (or -0, or NaN) goes to
 *     the left child 2n+1;
 *   - no input or output biases;
 *   - weights of K trees are stored [K, N, H], tree-major, rows of length H.
 *
 * Near-tie flag: |logit| < tie_rel * ||x_b||_2 * ||W_in[t,n]||_2.  A GPU path
 * may legitimately branch differently only at such a node.
 *
 * Around the layer (the intermediate layer of a pre-norm crammedBERT block,
 * Section 2.1): oracle_layer_norm gives the LayerNorm that feeds the FFF,
 * and oracle_round_bf16 the round-to-nearest-even storage of a result in
 * bf16; the residual sum itself is one addition, done by the caller.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_BF16 = 1, OR_F64 = 2 };
enum { OR_ACT_GELU_ERF = 0, OR_ACT_GELU_TANH = 1, OR_ACT_IDENTITY = 2 };

/* Exact widening of one stored element to double. */
static double widen_one(const void* base, int dtype, int64_t i) {
    if (dtype == OR_F32) return (double)((const float*)base)[i];
    if (dtype == OR_F64) return ((const double*)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static void widen_row(const void* base, int dtype, int64_t offset, int32_t h, double* out) {
    for (int32_t i = 0; i < h; ++i) out[i] = widen_one(base, dtype, offset + i);
}

/* GELU (Hendrycks and Gimpel): z * Phi(z) with Phi the standard normal CDF,
 * Phi(z) = (1 + erf(z / sqrt 2)) / 2.  The tanh form is their published
 * approximation; identity is a test-only activation. */
double oracle_activation(double z, int act) {
    if (act == OR_ACT_GELU_ERF) return 0.5 * z * (1.0 + erf(z / sqrt(2.0)));
    if (act == OR_ACT_GELU_TANH) {
        const double c = sqrt(2.0 / 3.14159265358979323846);
        return 0.5 * z * (1.0 + tanh(c * (z + 0.044715 * z * z * z)));
    }
    return z;
}

static double dot(const double* a, const double* b, int32_t h) {
    double s = 0.0;
    for (int32_t i = 0; i < h; ++i) s += a[i] * b[i];
    return s;
}

static double norm2(const double* a, int32_t h) { return sqrt(dot(a, a, h)); }

typedef struct {
    const void* x;
    int x_dtype;
    const void* w_in;
    const void* w_out;
    int w_dtype;
    int32_t hidden, depth, n_trees, act;
    double tie_rel;
    double* y;
    int32_t* nodes;
    double* logits;
    uint8_t* near_tie;
    int64_t b0, b1;
    int status;
} job_t;

static void* run_tokens(void* arg) {
    job_t* j = (job_t*)arg;
    const int32_t H = j->hidden, D = j->depth, T = j->n_trees;
    const int64_t N = ((int64_t)1 << (D + 1)) - 1;
    double* xr = (double*)malloc(sizeof(double) * (size_t)H);
    double* wr = (double*)malloc(sizeof(double) * (size_t)H);
    double* yr = (double*)malloc(sizeof(double) * (size_t)H);
    if (!xr || !wr || !yr) {
        j->status = -2;
        free(xr); free(wr); free(yr);
        return NULL;
    }
    for (int64_t b = j->b0; b < j->b1; ++b) {
        widen_row(j->x, j->x_dtype, b * H, H, xr);
        const double xnorm = norm2(xr, H);
        for (int32_t i = 0; i < H; ++i) yr[i] = 0.0;
        for (int32_t t = 0; t < T; ++t) {
            int64_t n = 0;
            for (int32_t l = 0; l <= D; ++l) {
                const int64_t row = ((int64_t)t * N + n) * H;
                widen_row(j->w_in, j->w_dtype, row, H, wr);
                const double logit = dot(xr, wr, H);
                const int64_t rec = (b * T + t) * (int64_t)(D + 1) + l;
                if (j->nodes) j->nodes[rec] = (int32_t)n;
                if (j->logits) j->logits[rec] = logit;
                if (j->near_tie)
                    j->near_tie[rec] = (uint8_t)(fabs(logit) < j->tie_rel * xnorm * norm2(wr, H));
                const double a = oracle_activation(logit, j->act);
                widen_row(j->w_out, j->w_dtype, row, H, wr);
                for (int32_t i = 0; i < H; ++i) yr[i] += a * wr[i];
                if (l < D) n = 2 * n + 1 + (logit > 0.0 ? 1 : 0);
            }
        }
        memcpy(j->y + b * H, yr, sizeof(double) * (size_t)H);
    }
    free(xr); free(wr); free(yr);
    return NULL;
}

static int check_common(const void* w_in, const void* w_out, int x_dtype, int w_dtype,
                        int32_t hidden, int32_t depth, int32_t n_trees, int act) {
    if (!w_in || !w_out) return -1;
    if ((x_dtype != OR_F32 && x_dtype != OR_BF16 && x_dtype != OR_F64) ||
        (w_dtype != OR_F32 && w_dtype != OR_BF16 && w_dtype != OR_F64))
        return -1;
    if (hidden < 1 || depth < 0 || depth > 30 || n_trees < 1) return -1;
    if (act < OR_ACT_GELU_ERF || act > OR_ACT_IDENTITY) return -1;
    return 0;
}

/* y[B,H] (double) = FFF(x); optional per-visit records nodes/logits/near_tie
 * laid out [B, T, D+1].  Tokens are split into contiguous ranges over
 * n_threads POSIX threads.  Returns 0, or -1 on bad arguments, -2 on
 * allocation failure. */
int oracle_forward(const void* x, int x_dtype, const void* w_in, const void* w_out, int w_dtype,
                   int64_t n_tokens, int32_t hidden, int32_t depth, int32_t n_trees, int act,
                   double tie_rel, double* y, int32_t* nodes, double* logits, uint8_t* near_tie,
                   int n_threads) {
    if (check_common(w_in, w_out, x_dtype, w_dtype, hidden, depth, n_trees, act)) return -1;
    if (n_tokens < 0) return -1;
    if (n_tokens == 0) return 0;
    if (!x || !y) return -1;
    if (n_threads < 1) n_threads = 1;
    if ((int64_t)n_threads > n_tokens) n_threads = (int)n_tokens;
    job_t* jobs = (job_t*)calloc((size_t)n_threads, sizeof(job_t));
    pthread_t* tids = (pthread_t*)calloc((size_t)n_threads, sizeof(pthread_t));
    if (!jobs || !tids) {
        free(jobs); free(tids);
        return -2;
    }
    int status = 0;
    for (int k = 0; k < n_threads; ++k) {
        job_t* j = &jobs[k];
        j->x = x; j->x_dtype = x_dtype; j->w_in = w_in; j->w_out = w_out; j->w_dtype = w_dtype;
        j->hidden = hidden; j->depth = depth; j->n_trees = n_trees; j->act = act;
        j->tie_rel = tie_rel; j->y = y; j->nodes = nodes; j->logits = logits; j->near_tie = near_tie;
        j->b0 = n_tokens * k / n_threads;
        j->b1 = n_tokens * (k + 1) / n_threads;
    }
    int started = 0;
    for (int k = 1; k < n_threads; ++k) {
        if (pthread_create(&tids[k], NULL, run_tokens, &jobs[k]) != 0) {
            jobs[k].status = -2;
            break;
        }
        started = k;
    }
    run_tokens(&jobs[0]);
    for (int k = 1; k <= started; ++k) pthread_join(tids[k], NULL);
    for (int k = 0; k < n_threads; ++k)
        if (jobs[k].status) status = jobs[k].status;
    free(jobs); free(tids);
    return status;
}

/* Output of one token along a GIVEN path per tree, path laid out [T, D+1].
 * The path must start at the root and step to a child each level (any child:
 * the signs are not checked, so a path that took the other branch at a near
 * tie can be evaluated).  Returns 0, -1 on bad arguments, -3 if the path is
 * not a root-to-leaf walk. */
int oracle_eval_path(const void* x_row, int x_dtype, const void* w_in, const void* w_out, int w_dtype,
                     int32_t hidden, int32_t depth, int32_t n_trees, int act, const int32_t* path,
                     double* y_row, double* logits) {
    if (check_common(w_in, w_out, x_dtype, w_dtype, hidden, depth, n_trees, act)) return -1;
    if (!x_row || !path || !y_row) return -1;
    const int32_t H = hidden, D = depth, T = n_trees;
    const int64_t N = ((int64_t)1 << (D + 1)) - 1;
    for (int32_t t = 0; t < T; ++t) {
        const int32_t* p = path + (int64_t)t * (D + 1);
        if (p[0] != 0) return -3;
        for (int32_t l = 1; l <= D; ++l) {
            const int64_t parent = p[l - 1], child = p[l];
            if (child != 2 * parent + 1 && child != 2 * parent + 2) return -3;
        }
    }
    double* xr = (double*)malloc(sizeof(double) * (size_t)H);
    double* wr = (double*)malloc(sizeof(double) * (size_t)H);
    if (!xr || !wr) {
        free(xr); free(wr);
        return -2;
    }
    widen_row(x_row, x_dtype, 0, H, xr);
    for (int32_t i = 0; i < H; ++i) y_row[i] = 0.0;
    for (int32_t t = 0; t < T; ++t) {
        for (int32_t l = 0; l <= D; ++l) {
            const int64_t n = path[(int64_t)t * (D + 1) + l];
            const int64_t row = ((int64_t)t * N + n) * H;
            widen_row(w_in, w_dtype, row, H, wr);
            const double logit = dot(xr, wr, H);
            if (logits) logits[(int64_t)t * (D + 1) + l] = logit;
            const double a = oracle_activation(logit, act);
            widen_row(w_out, w_dtype, row, H, wr);
            for (int32_t i = 0; i < H; ++i) y_row[i] += a * wr[i];
        }
    }
    free(xr); free(wr);
    return 0;
}

/* LayerNorm of every row of x[B,H] (Ba, Kiros and Hinton): with the row mean
 * mu = sum_i x_i / H and the biased variance var = sum_i (x_i - mu)^2 / H,
 * out_i = (x_i - mu) / sqrt(var + eps) * gamma_i + beta_i.  gamma and beta
 * may be NULL (ones and zeros).  Two passes over each row, in fp64.  Returns
 * 0, or -1 on bad arguments. */
int oracle_layer_norm(const void* x, int x_dtype, int64_t n_tokens, int32_t hidden, const double* gamma,
                      const double* beta, double eps, double* out) {
    if (!x || !out || n_tokens < 0 || hidden < 1 || !(eps >= 0.0)) return -1;
    if (x_dtype != OR_F32 && x_dtype != OR_BF16 && x_dtype != OR_F64) return -1;
    const int32_t H = hidden;
    for (int64_t b = 0; b < n_tokens; ++b) {
        double* o = out + b * H;
        widen_row(x, x_dtype, b * H, H, o);
        double mu = 0.0;
        for (int32_t i = 0; i < H; ++i) mu += o[i];
        mu /= H;
        double var = 0.0;
        for (int32_t i = 0; i < H; ++i) var += (o[i] - mu) * (o[i] - mu);
        var /= H;
        const double inv = 1.0 / sqrt(var + eps);
        for (int32_t i = 0; i < H; ++i) {
            double v = (o[i] - mu) * inv;
            if (gamma) v *= gamma[i];
            if (beta) v += beta[i];
            o[i] = v;
        }
    }
    return 0;
}

/* bf16 storage of doubles: the bf16 value nearest to v (ties to the even
 * significand), returned as its 16-bit pattern.  bf16 has fp32's exponent
 * range and 8 significant bits, so for |v| = m * 2^e with m in [0.5, 1) the
 * spacing is 2^(e-8), or 2^-133 below the normal range.  Values past the
 * largest finite bf16 by half a spacing or more become infinities. */
int oracle_round_bf16(const double* in, int64_t n, uint16_t* out) {
    if ((!in || !out) && n > 0) return -1;
    for (int64_t k = 0; k < n; ++k) {
        const double v = in[k];
        double r = v;
        if (v != 0.0 && isfinite(v)) {
            int e;
            frexp(v, &e);
            int q = e - 8;
            if (q < -133) q = -133;
            r = ldexp(nearbyint(ldexp(v, -q)), q);  /* default rounding mode: ties to even */
            if (fabs(r) > 3.3895313892515355e38) r = v > 0 ? INFINITY : -INFINITY;
        }
        const float f = (float)r;  /* exact: r has at most 8 significant bits */
        uint32_t bits;
        memcpy(&bits, &f, sizeof bits);
        if (isnan(v)) bits = 0x7FC00000u;
        out[k] = (uint16_t)(bits >> 16);
    }
    return 0;
}

/* d act / dz: GELU'(z) = Phi(z) + z phi(z) with phi the standard normal
 * density; the tanh form's derivative follows from d tanh(u) = 1 - tanh(u)^2;
 * identity: 1. */
double oracle_activation_grad(double z, int act) {
    if (act == OR_ACT_GELU_ERF)
        return 0.5 * (1.0 + erf(z / sqrt(2.0))) + z * exp(-0.5 * z * z) / sqrt(2.0 * 3.14159265358979323846);
    if (act == OR_ACT_GELU_TANH) {
        const double c = sqrt(2.0 / 3.14159265358979323846);
        const double u = c * (z + 0.044715 * z * z * z);
        const double t = tanh(u);
        return 0.5 * (1.0 + t) + 0.5 * z * (1.0 - t * t) * c * (1.0 + 3.0 * 0.044715 * z * z);
    }
    return 1.0;
}

/* Backward of the layer with the routing held fixed (hard routing): the tree
 * walk's branch decisions are not differentiable, so gradients flow only
 * through the D+1 visited nodes of every (token, tree).  With the given path
 * n_l, logits l_l = <x_b, W_in[t,n_l]> and a_l = act(l_l), y_b = sum a_l
 * W_out[t,n_l], and the upstream gradient dy_b:
 *   dW_out[t,n_l] += a_l dy_b
 *   da_l           = <dy_b, W_out[t,n_l]>
 *   dl_l           = da_l act'(l_l)
 *   dW_in[t,n_l]  += dl_l x_b
 *   dx_b          += dl_l W_in[t,n_l]
 * path is [B, T, D+1] and must be root-to-leaf walks; dy, dx are [B,H] and
 * dw_in, dw_out [T,N,H], all double, overwritten (rows off every path are
 * zero); dx, dw_in or dw_out may be NULL.  The logits are recomputed here
 * from x and W_in.  Single-threaded.  Returns 0, -1 on bad arguments, -2 on
 * allocation failure, -3 if a path is not a root-to-leaf walk. */
int oracle_backward(const void* x, int x_dtype, const void* w_in, const void* w_out, int w_dtype,
                    const double* dy, const int32_t* path, int64_t n_tokens, int32_t hidden, int32_t depth,
                    int32_t n_trees, int act, double* dx, double* dw_in, double* dw_out) {
    if (check_common(w_in, w_out, x_dtype, w_dtype, hidden, depth, n_trees, act)) return -1;
    if (n_tokens < 0 || ((!x || !dy || !path) && n_tokens > 0)) return -1;
    const int32_t H = hidden, D = depth, T = n_trees;
    const int64_t N = ((int64_t)1 << (D + 1)) - 1;
    for (int64_t b = 0; b < n_tokens; ++b)
        for (int32_t t = 0; t < T; ++t) {
            const int32_t* p = path + (b * T + t) * (D + 1);
            if (p[0] != 0) return -3;
            for (int32_t l = 1; l <= D; ++l)
                if (p[l] != 2 * p[l - 1] + 1 && p[l] != 2 * p[l - 1] + 2) return -3;
        }
    if (dw_in) memset(dw_in, 0, sizeof(double) * (size_t)(T * N * H));
    if (dw_out) memset(dw_out, 0, sizeof(double) * (size_t)(T * N * H));
    double* xr = (double*)malloc(sizeof(double) * (size_t)H);
    double* wi = (double*)malloc(sizeof(double) * (size_t)H);
    double* wo = (double*)malloc(sizeof(double) * (size_t)H);
    if (!xr || !wi || !wo) {
        free(xr); free(wi); free(wo);
        return -2;
    }
    for (int64_t b = 0; b < n_tokens; ++b) {
        widen_row(x, x_dtype, b * H, H, xr);
        const double* g = dy + b * H;
        double* dxr = dx ? dx + b * H : NULL;
        if (dxr)
            for (int32_t i = 0; i < H; ++i) dxr[i] = 0.0;
        for (int32_t t = 0; t < T; ++t) {
            const int32_t* p = path + (b * T + t) * (D + 1);
            for (int32_t l = 0; l <= D; ++l) {
                const int64_t row = ((int64_t)t * N + p[l]) * H;
                widen_row(w_in, w_dtype, row, H, wi);
                widen_row(w_out, w_dtype, row, H, wo);
                const double logit = dot(xr, wi, H);
                const double a = oracle_activation(logit, act);
                const double dl = dot(g, wo, H) * oracle_activation_grad(logit, act);
                for (int32_t i = 0; i < H; ++i) {
                    if (dw_out) dw_out[row + i] += a * g[i];
                    if (dw_in) dw_in[row + i] += dl * xr[i];
                    if (dxr) dxr[i] += dl * wi[i];
                }
            }
        }
    }
    free(xr); free(wi); free(wo);
    return 0;
}
