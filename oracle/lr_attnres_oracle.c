/*
 * fp64 CPU oracle for the depth-wise residual routing of Low-Rank Attention
 * Residuals (LR-AttnRes), arXiv 2607.09694.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the routing computes.  It is linked only by the test
 * suite, by the smoke check and by the CPU-baseline leg of the benchmark.
 * The GPU library never includes, links or calls it, and it shares no code,
 * header, table or constant with the GPU library.
 *
 * What it follows (Section 3 of the paper, "Method"):
 *   - Eq. (lr_source_pair): source i is a pair (o_i in R^d, k_i in R^r).
 *   - Eq. (lr_key_norm): kbar_i = RMSNorm(k_i); parameter-free RMSNorm
 *     (Appendix A, "Parameters": the paper's RMSNorm convention has no gain),
 *     rho_i = sqrt(mean_j k_ij^2 + eps), kbar_i = k_i / rho_i.
 *   - Eq. (lr_attnres_weight): alpha_i = softmax over sources of q^T kbar_i.
 *   - Eq. (lr_attnres_output): h = sum_i alpha_i o_i.
 *   - Projected keys (Sec. 3.3, Eq. fused_projection): k_i is a separate
 *     input tensor K[S][N][r].
 *   - Sliced keys (Sec. 3.4, Eq. sliced_key): k_i = tail_r(o_i), the last r
 *     coordinates of the value (1-based d-r+1..d, 0-based [d-r, d)).
 *   - Full-rank AttnRes (Sec. 3.1, Eqs. attnres_weight / attnres_output):
 *     the key is the whole value, r = d; Sec. 3.4 states that sliced keys
 *     with r = d reduce to it.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - eps: never stated; it is an explicit argument added to the mean of
 *     squares inside the square root.
 *   - The softmax subtracts the per-token maximum score first; this is an
 *     identity of the softmax, not an approximation.
 *   - Source order is the stack order i = 0 (embedding) .. S-1.
 *   - The backward pass is not stated by the paper; it is derived here by
 *     hand for the scalar loss L = sum_n dH[n] . h[n]:
 *         g_i   = dH . o_i
 *         ds_i  = alpha_i (g_i - sum_l alpha_l g_l)        (softmax)
 *         dV_i  = alpha_i dH                               (value path)
 *         dk_i  = (ds_i / rho_i) (q - kbar_i s_i / r)      (RMSNorm, s_i = q.kbar_i)
 *         dq    = sum_n sum_i ds_i kbar_i
 *     With sliced keys dk_i is added into the last r coordinates of dV_i,
 *     with full-rank keys into all d coordinates (the key is the value).
 *     The forward is pinned by closed-form cases and invariants, the
 *     backward by central finite differences of this same forward.
 *
 * Arithmetic: every input is widened exactly to double (bf16 by placing its
 * 16 bits in the high half of an IEEE single, fp32 by conversion), and every
 * operation is done in double.  Outputs are double and unrounded.
 *
 * Storage codes for V, K and dH: 0 = fp32, 1 = bf16 (raw uint16 bits),
 * 2 = fp64.  Key modes: 0 = projected, 1 = sliced, 2 = full-rank.
 * q and eps are passed as double (callers widen the fp32 values exactly).
 *
 * Token ranges: each call computes tokens n in [n0, n1) of a problem whose
 * inputs are the complete [S][N][.] stacks; outputs hold only that range.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_STORE_F32 = 0, ORC_STORE_BF16 = 1, ORC_STORE_F64 = 2 };
enum { ORC_KEYS_PROJECTED = 0, ORC_KEYS_SLICED = 1, ORC_KEYS_FULL = 2 };

struct orc_problem {
    const void *V;   /* [S][N][d] values o_i            */
    const void *K;   /* [S][N][r] projected keys or NULL */
    const double *q; /* [r] pseudo-query                 */
    long long S, N, d, r;
    int mode, store;
    double eps;
};

/* Exact widening of one stored element to double. */
static double widen(const void *base, int store, long long idx)
{
    if (store == ORC_STORE_F32)
        return (double)((const float *)base)[idx];
    if (store == ORC_STORE_F64)
        return ((const double *)base)[idx];
    {
        uint32_t bits = (uint32_t)((const uint16_t *)base)[idx] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
}

/* o_i[j] for token n: V[i][n][j]. */
static double value_elem(const struct orc_problem *p, long long i, long long n, long long j)
{
    return widen(p->V, p->store, (i * p->N + n) * p->d + j);
}

/* k_i[j] for token n, per the key mode (Eq. fused_projection / sliced_key /
 * attnres_weight). */
static double key_elem(const struct orc_problem *p, long long i, long long n, long long j)
{
    if (p->mode == ORC_KEYS_PROJECTED)
        return widen(p->K, p->store, (i * p->N + n) * p->r + j);
    if (p->mode == ORC_KEYS_SLICED)
        return value_elem(p, i, n, p->d - p->r + j);
    return value_elem(p, i, n, j);
}

/* Eq. lr_key_norm: rho_i = sqrt(mean_j k_ij^2 + eps), kbar_i = k_i / rho_i.
 * Then the score s_i = q^T kbar_i (Eq. lr_attnres_weight).
 * kbar is [S][r]; rho and s are [S]. */
static void normalised_keys_and_scores(const struct orc_problem *p, long long n,
                                       double *kbar, double *rho, double *s)
{
    for (long long i = 0; i < p->S; ++i) {
        double sumsq = 0.0;
        for (long long j = 0; j < p->r; ++j) {
            double k = key_elem(p, i, n, j);
            sumsq += k * k;
        }
        rho[i] = sqrt(sumsq / (double)p->r + p->eps);
        s[i] = 0.0;
        for (long long j = 0; j < p->r; ++j) {
            kbar[i * p->r + j] = key_elem(p, i, n, j) / rho[i];
            s[i] += p->q[j] * kbar[i * p->r + j];
        }
    }
}

/* Eq. lr_attnres_weight: alpha = softmax over the sources of the scores. */
static void depth_softmax(long long S, const double *s, double *alpha)
{
    double m = s[0];
    for (long long i = 1; i < S; ++i)
        if (s[i] > m)
            m = s[i];
    double z = 0.0;
    for (long long i = 0; i < S; ++i) {
        alpha[i] = exp(s[i] - m);
        z += alpha[i];
    }
    for (long long i = 0; i < S; ++i)
        alpha[i] /= z;
}

static int check_problem(const struct orc_problem *p, long long n0, long long n1)
{
    if (p->S < 1 || p->N < 0 || p->d < 1 || p->r < 1)
        return 1;
    if (n0 < 0 || n1 < n0 || n1 > p->N)
        return 1;
    if (p->mode == ORC_KEYS_PROJECTED && p->K == NULL)
        return 1;
    if (p->mode == ORC_KEYS_SLICED && p->r > p->d)
        return 1;
    if (p->mode == ORC_KEYS_FULL && p->r != p->d)
        return 1;
    if (p->mode < 0 || p->mode > 2 || p->store < 0 || p->store > 2)
        return 1;
    return 0;
}

/* Scratch for one token: kbar[S*r], rho[S], s[S], alpha[S], g[S], ds[S]. */
static double *token_scratch(const struct orc_problem *p)
{
    return (double *)malloc(sizeof(double) * (size_t)(p->S * p->r + 5 * p->S));
}

/* Softmax weights alpha[n - n0][i] for tokens in [n0, n1). */
int orc_route_weights(const void *V, const void *K, const double *q, double *alpha,
                      long long S, long long N, long long d, long long r,
                      int mode, int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || alpha == NULL || q == NULL || V == NULL)
        return 1;
    int failed = 0;
#pragma omp parallel
    {
        double *w = token_scratch(&p);
        if (w == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (long long n = n0; n < n1; ++n) {
            if (w == NULL)
                continue;
            double *kbar = w, *rho = kbar + S * r, *s = rho + S;
            normalised_keys_and_scores(&p, n, kbar, rho, s);
            depth_softmax(S, s, alpha + (n - n0) * S);
        }
        free(w);
    }
    return failed;
}

/* Forward, Eq. lr_attnres_output: H[n - n0][:] = sum_i alpha_i o_i. */
int orc_route_fwd(const void *V, const void *K, const double *q, double *H,
                  long long S, long long N, long long d, long long r,
                  int mode, int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || H == NULL || q == NULL || V == NULL)
        return 1;
    int failed = 0;
#pragma omp parallel
    {
        double *w = token_scratch(&p);
        if (w == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (long long n = n0; n < n1; ++n) {
            if (w == NULL)
                continue;
            double *kbar = w, *rho = kbar + S * r, *s = rho + S, *alpha = s + S;
            normalised_keys_and_scores(&p, n, kbar, rho, s);
            depth_softmax(S, s, alpha);
            double *h = H + (n - n0) * d;
            for (long long j = 0; j < d; ++j) {
                double acc = 0.0;
                for (long long i = 0; i < S; ++i)
                    acc += alpha[i] * value_elem(&p, i, n, j);
                h[j] = acc;
            }
        }
        free(w);
    }
    return failed;
}

/* Backward of L = sum_n dH[n] . h[n] (derived; see the file header).
 *   dV [S][n1-n0][d]   gradient w.r.t. the values, including the key path for
 *                      sliced and full-rank keys (the key is part of the value)
 *   dK [S][n1-n0][r]   gradient w.r.t. projected keys (projected mode only;
 *                      must be NULL otherwise)
 *   dq [r]             gradient w.r.t. q summed over tokens [n0, n1)
 * dH is [N][d] in the same storage as V; row n is token n. */
int orc_route_bwd(const void *V, const void *K, const double *q, const void *dH,
                  double *dV, double *dK, double *dq,
                  long long S, long long N, long long d, long long r,
                  int mode, int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || q == NULL || V == NULL || dH == NULL || dV == NULL ||
        dq == NULL)
        return 1;
    if ((mode == ORC_KEYS_PROJECTED) != (dK != NULL))
        return 1;
    const long long nt = n1 - n0;
    /* Per-token dq contributions are summed in token order after each block,
     * so the result does not depend on the thread count. */
    const long long block = 256;
    double *dq_tok = (double *)malloc(sizeof(double) * (size_t)(block * r));
    if (dq_tok == NULL)
        return 1;
    for (long long j = 0; j < r; ++j)
        dq[j] = 0.0;
    int failed = 0;
    for (long long b0 = n0; b0 < n1; b0 += block) {
        long long b1 = b0 + block < n1 ? b0 + block : n1;
#pragma omp parallel
        {
            double *w = token_scratch(&p);
            if (w == NULL) {
#pragma omp atomic write
                failed = 1;
            }
#pragma omp for schedule(static)
            for (long long n = b0; n < b1; ++n) {
                if (w == NULL)
                    continue;
                double *kbar = w, *rho = kbar + S * r, *s = rho + S, *alpha = s + S;
                double *g = alpha + S, *ds = g + S;
                normalised_keys_and_scores(&p, n, kbar, rho, s);
                depth_softmax(S, s, alpha);
                /* g_i = dH . o_i and the softmax gradient. */
                double gbar = 0.0;
                for (long long i = 0; i < S; ++i) {
                    g[i] = 0.0;
                    for (long long j = 0; j < d; ++j)
                        g[i] += widen(dH, store, n * d + j) * value_elem(&p, i, n, j);
                    gbar += alpha[i] * g[i];
                }
                for (long long i = 0; i < S; ++i)
                    ds[i] = alpha[i] * (g[i] - gbar);
                /* Value path: dV_i = alpha_i dH. */
                for (long long i = 0; i < S; ++i)
                    for (long long j = 0; j < d; ++j)
                        dV[(i * nt + (n - n0)) * d + j] = alpha[i] * widen(dH, store, n * d + j);
                /* Key path through the score and the RMSNorm. */
                for (long long i = 0; i < S; ++i) {
                    for (long long j = 0; j < r; ++j) {
                        double dk = ds[i] / rho[i] *
                                    (q[j] - kbar[i * r + j] * s[i] / (double)r);
                        if (mode == ORC_KEYS_PROJECTED)
                            dK[(i * nt + (n - n0)) * r + j] = dk;
                        else if (mode == ORC_KEYS_SLICED)
                            dV[(i * nt + (n - n0)) * d + (d - r) + j] += dk;
                        else
                            dV[(i * nt + (n - n0)) * d + j] += dk;
                    }
                }
                /* dq contribution of this token: sum_i ds_i kbar_i. */
                double *dqt = dq_tok + (n - b0) * r;
                for (long long j = 0; j < r; ++j) {
                    dqt[j] = 0.0;
                    for (long long i = 0; i < S; ++i)
                        dqt[j] += ds[i] * kbar[i * r + j];
                }
            }
            free(w);
        }
        for (long long n = b0; n < b1; ++n)
            for (long long j = 0; j < r; ++j)
                dq[j] += dq_tok[(n - b0) * r + j];
    }
    free(dq_tok);
    return failed;
}

/* ---------------------------------------------------------------------------
 * Block sources (Sec. 3.1 "Block AttnRes", Eqs. block_attnres_sum and
 * block_attnres_partial_sum, with the low-rank keys of Sec. 3.2).
 *
 * The 2L residual-writing sub-layers are grouped into consecutive blocks of
 * c outputs: block j (1-based) holds outputs (j-1)c+1 .. jc.  Site t reads
 * the embedding o_0, every completed block summary b_j = sum of its members,
 * and the partial summary of the block in progress if it has members.
 * Reading where the paper is silent: a summary's key is the sum of its
 * members' keys.  For sliced keys that is exactly the tail of the summed
 * value; for projected keys it is the key part of the summed [o_i; k_i].
 * ------------------------------------------------------------------------- */

/* Number of sources at site t >= 1 with blocks of c outputs:
 * 1 + floor((t-1)/c) completed-or-current blocks, counting a non-empty
 * partial block. */
long long orc_block_num_sources(long long t, long long c)
{
    if (t < 1 || c < 1)
        return -1;
    return 1 + (t - 1) / c + ((t - 1) % c != 0);
}

/* Slot of output i: 0 for the embedding, block ceil(i / c) otherwise. */
static long long block_slot(long long i, long long c) { return i == 0 ? 0 : (i - 1) / c + 1; }

/* The block summaries site t reads (Sec. 3.1, Eqs. block_attnres_sum and
 * block_attnres_partial_sum), exact in double: slot 0 is the embedding o_0,
 * slot j >= 1 the sum of the outputs of block j written before site t (the
 * last slot may be partial).  B [S][nt][d] and KB [S][nt][r] (projected keys;
 * else NULL) must be zero on entry; tokens [n0, n1), nt = n1 - n0. */
static void block_sums(const void *O, const void *KO, double *B, double *KB, long long t,
                       long long c, long long N, long long d, long long r, int store,
                       long long n0, long long n1)
{
    const long long nt = n1 - n0;
    for (long long i = 0; i < t; ++i) {
        /* output i belongs to slot 0 (embedding) or block ceil(i / c) */
        const long long slot = block_slot(i, c);
        for (long long n = n0; n < n1; ++n) {
            for (long long j = 0; j < d; ++j)
                B[(slot * nt + (n - n0)) * d + j] += widen(O, store, (i * N + n) * d + j);
            if (KB)
                for (long long j = 0; j < r; ++j)
                    KB[(slot * nt + (n - n0)) * r + j] += widen(KO, store, (i * N + n) * r + j);
        }
    }
}

static int block_args_ok(const void *O, const void *KO, long long S, long long N, long long d,
                         long long r, int mode, int store, long long n0, long long n1)
{
    return S >= 1 && N >= 0 && d >= 1 && r >= 1 && n0 >= 0 && n1 >= n0 && n1 <= N &&
           O != NULL && (mode == ORC_KEYS_PROJECTED || mode == ORC_KEYS_SLICED) &&
           (mode == ORC_KEYS_PROJECTED) == (KO != NULL) &&
           !(mode == ORC_KEYS_SLICED && r > d) && store >= 0 && store <= 2;
}

/* The summaries themselves (see block_sums): B [S][n1-n0][d], KB
 * [S][n1-n0][r] for projected keys (else NULL), S = orc_block_num_sources(t, c).
 * O is [t][N][d] (o_0 .. o_{t-1}), KO [t][N][r] or NULL. */
int orc_block_summaries(const void *O, const void *KO, double *B, double *KB, long long t,
                        long long c, long long N, long long d, long long r, int mode,
                        int store, long long n0, long long n1)
{
    const long long S = orc_block_num_sources(t, c);
    if (!block_args_ok(O, KO, S, N, d, r, mode, store, n0, n1) || B == NULL ||
        (mode == ORC_KEYS_PROJECTED) != (KB != NULL))
        return 1;
    const long long nt = n1 - n0;
    memset(B, 0, sizeof(double) * (size_t)(S * nt * d));
    if (KB)
        memset(KB, 0, sizeof(double) * (size_t)(S * nt * r));
    block_sums(O, KO, B, KB, t, c, N, d, r, store, n0, n1);
    return 0;
}

/* Forward at site t: O is [t][N][d] (o_0 .. o_{t-1}), KO is [t][N][r]
 * (projected keys) or NULL.  H[n - n0][:] as in orc_route_fwd, with the
 * block summaries of the outputs as sources, for tokens [n0, n1).  The
 * summaries are formed in double; then the routing of Sec. 3.2 applies to
 * them unchanged (sliced keys: the tail of each summary). */
int orc_block_route_fwd(const void *O, const void *KO, const double *q, double *H,
                        long long t, long long c, long long N, long long d, long long r,
                        int mode, int store, double eps, long long n0, long long n1)
{
    const long long S = orc_block_num_sources(t, c);
    if (!block_args_ok(O, KO, S, N, d, r, mode, store, n0, n1) || q == NULL || H == NULL)
        return 1;
    const long long nt = n1 - n0;
    /* Summaries of the token range, double: B [S][nt][d], KB [S][nt][r]. */
    double *B = (double *)calloc((size_t)(S * nt * d), sizeof(double));
    double *KB = mode == ORC_KEYS_PROJECTED ? (double *)calloc((size_t)(S * nt * r), sizeof(double))
                                            : NULL;
    if (B == NULL || (mode == ORC_KEYS_PROJECTED && KB == NULL)) {
        free(B);
        free(KB);
        return 1;
    }
    block_sums(O, KO, B, KB, t, c, N, d, r, store, n0, n1);
    const int rc = orc_route_fwd(B, KB, q, H, S, nt, d, r, mode, ORC_STORE_F64, eps, 0, nt);
    free(B);
    free(KB);
    return rc;
}

/* Backward of the block-source forward at site t for L = sum_n dH[n] . h[n]:
 * the routing backward (orc_route_bwd) applied to the block summaries gives
 * each summary's gradient; since a summary is the plain sum of its members,
 * every member's output (and projected key) receives its summary's gradient
 * unchanged.  dO is [t][n1-n0][d], dKO [t][n1-n0][r] (projected only, else
 * NULL), dq [r] summed over tokens [n0, n1); dH is [N][d] in O's storage. */
int orc_block_route_bwd(const void *O, const void *KO, const double *q, const void *dH,
                        double *dO, double *dKO, double *dq, long long t, long long c,
                        long long N, long long d, long long r, int mode, int store, double eps,
                        long long n0, long long n1)
{
    const long long S = orc_block_num_sources(t, c);
    if (S < 1 || N < 0 || d < 1 || r < 1 || n0 < 0 || n1 < n0 || n1 > N || O == NULL ||
        q == NULL || dH == NULL || dO == NULL || dq == NULL ||
        (mode != ORC_KEYS_PROJECTED && mode != ORC_KEYS_SLICED) ||
        (mode == ORC_KEYS_PROJECTED) != (KO != NULL) ||
        (mode == ORC_KEYS_PROJECTED) != (dKO != NULL) || (mode == ORC_KEYS_SLICED && r > d) ||
        store < 0 || store > 2)
        return 1;
    const long long nt = n1 - n0;
    const int proj = mode == ORC_KEYS_PROJECTED;
    double *B = (double *)calloc((size_t)(S * nt * d), sizeof(double));
    double *KB = proj ? (double *)calloc((size_t)(S * nt * r), sizeof(double)) : NULL;
    double *dHr = (double *)malloc(sizeof(double) * (size_t)(nt * d));
    double *dB = (double *)malloc(sizeof(double) * (size_t)(S * nt * d));
    double *dKB = proj ? (double *)malloc(sizeof(double) * (size_t)(S * nt * r)) : NULL;
    int rc = 1;
    if (B == NULL || dHr == NULL || dB == NULL || (proj && (KB == NULL || dKB == NULL)))
        goto done;
    block_sums(O, KO, B, KB, t, c, N, d, r, store, n0, n1);
    for (long long n = n0; n < n1; ++n)
        for (long long j = 0; j < d; ++j)
            dHr[(n - n0) * d + j] = widen(dH, store, n * d + j);
    rc = orc_route_bwd(B, KB, q, dHr, dB, dKB, dq, S, nt, d, r, mode, ORC_STORE_F64, eps, 0, nt);
    if (rc)
        goto done;
    for (long long i = 0; i < t; ++i) {
        const long long slot = block_slot(i, c);
        memcpy(dO + i * nt * d, dB + slot * nt * d, sizeof(double) * (size_t)(nt * d));
        if (proj)
            memcpy(dKO + i * nt * r, dKB + slot * nt * r, sizeof(double) * (size_t)(nt * r));
    }
done:
    free(B);
    free(KB);
    free(dHr);
    free(dB);
    free(dKB);
    return rc;
}

/* Online-softmax state of the routing over a set of sources (Sec. 3.5: the
 * two-phase inference merges inter-block and intra-block results with an
 * online-softmax update).  For each token in [n0, n1), over the S sources
 * given (same layout and key modes as orc_route_fwd):
 *   M[n]      = max_i s_i
 *   Lsum[n]   = sum_i exp(s_i - M[n])
 *   ACC[n][:] = sum_i exp(s_i - M[n]) o_i
 * so that ACC / Lsum is orc_route_fwd over the same sources. */
int orc_route_state(const void *V, const void *K, const double *q, double *Mx, double *Lsum,
                    double *ACC, long long S, long long N, long long d, long long r, int mode,
                    int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || Mx == NULL || Lsum == NULL || ACC == NULL || q == NULL ||
        V == NULL)
        return 1;
    int failed = 0;
#pragma omp parallel
    {
        double *w = token_scratch(&p);
        if (w == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (long long n = n0; n < n1; ++n) {
            if (w == NULL)
                continue;
            double *kbar = w, *rho = kbar + S * r, *s = rho + S;
            normalised_keys_and_scores(&p, n, kbar, rho, s);
            double m = s[0];
            for (long long i = 1; i < S; ++i)
                if (s[i] > m)
                    m = s[i];
            double l = 0.0;
            double *acc = ACC + (n - n0) * d;
            for (long long j = 0; j < d; ++j)
                acc[j] = 0.0;
            for (long long i = 0; i < S; ++i) {
                const double e = exp(s[i] - m);
                l += e;
                for (long long j = 0; j < d; ++j)
                    acc[j] += e * value_elem(&p, i, n, j);
            }
            Mx[n - n0] = m;
            Lsum[n - n0] = l;
        }
        free(w);
    }
    return failed;
}

/* Eq. effective_sources (Sec. 4.5, "Effective number of sources"): the
 * perplexity of the routing distribution, exp(-sum_i alpha_i log alpha_i).
 * Terms with alpha_i = 0 (possible only after underflow) contribute their
 * limit 0. */
static double effective_sources(long long S, const double *alpha)
{
    double ent = 0.0;
    for (long long i = 0; i < S; ++i)
        if (alpha[i] > 0.0)
            ent -= alpha[i] * log(alpha[i]);
    return exp(ent);
}

/* N_eff[n - n0] of the routing over the S sources (same arguments as
 * orc_route_weights). */
int orc_effective_sources(const void *V, const void *K, const double *q, double *NEFF,
                          long long S, long long N, long long d, long long r, int mode,
                          int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || NEFF == NULL || q == NULL || V == NULL)
        return 1;
    int failed = 0;
#pragma omp parallel
    {
        double *w = token_scratch(&p);
        if (w == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(static)
        for (long long n = n0; n < n1; ++n) {
            if (w == NULL)
                continue;
            double *kbar = w, *rho = kbar + S * r, *s = rho + S, *alpha = s + S;
            normalised_keys_and_scores(&p, n, kbar, rho, s);
            depth_softmax(S, s, alpha);
            NEFF[n - n0] = effective_sources(S, alpha);
        }
        free(w);
    }
    return failed;
}

/* Every read site of a model pass from one stack of sources (Sec. 3.1, Eq.
 * full_attnres_source_set: site t reads the sources 0 .. t-1).  Site j = 0 .. T-1 reads the first first+j sources of the
 * [S][N][.] stacks with its own query Q[j][0..r) and gives
 *   H[j][n - n0][:]  = its routed state (Eq. lr_attnres_output),
 *   NEFF[j][n - n0]  = its effective number of sources (Eq. effective_sources;
 *                      NEFF may be NULL).
 * Requires 1 <= first and first + T - 1 <= S.  Each site is the single-site
 * routing of that prefix: the stacks are source-major, so the first S'
 * sources of an [S][N][.] stack are themselves an [S'][N][.] stack. */
int orc_route_all_fwd(const void *V, const void *K, const double *Q, double *H, double *NEFF,
                      long long S, long long N, long long d, long long r, long long first,
                      long long T, int mode, int store, double eps, long long n0, long long n1)
{
    struct orc_problem p = {V, K, Q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || H == NULL || Q == NULL || V == NULL)
        return 1;
    if (first < 1 || T < 1 || first + T - 1 > S)
        return 1;
    const long long nt = n1 - n0;
    int failed = 0;
#pragma omp parallel
    {
        double *w = token_scratch(&p);
        if (w == NULL) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for collapse(2) schedule(static)
        for (long long j = 0; j < T; ++j) {
            for (long long n = n0; n < n1; ++n) {
                if (w == NULL)
                    continue;
                struct orc_problem site = p;
                site.S = first + j;
                site.q = Q + j * r;
                double *kbar = w, *rho = kbar + S * r, *s = rho + S, *alpha = s + S;
                normalised_keys_and_scores(&site, n, kbar, rho, s);
                depth_softmax(site.S, s, alpha);
                double *h = H + (j * nt + (n - n0)) * d;
                for (long long c = 0; c < d; ++c) {
                    double acc = 0.0;
                    for (long long i = 0; i < site.S; ++i)
                        acc += alpha[i] * value_elem(&site, i, n, c);
                    h[c] = acc;
                }
                if (NEFF)
                    NEFF[j * nt + (n - n0)] = effective_sources(site.S, alpha);
            }
        }
        free(w);
    }
    return failed;
}

/* Backward of every read site of a pass (the gradient of orc_route_all_fwd;
 * the paper states no backward).  For the loss
 *   L = sum_j sum_n dH[j][n] . h_j[n],
 * site j's routed state h_j depends on the first first+j sources and on its
 * own query Q[j] only, so dL/dV and dL/dK are the sums over sites of each
 * site's single-site gradient (orc_route_bwd over that prefix with dH[j]),
 * and dL/dQ[j] is site j's dq.  Outputs, for tokens n in [n0, n1):
 *   dV[i][n - n0][:]  for every source i < S (zero for a source no site reads),
 *   dK[i][n - n0][:]  likewise (projected keys; NULL otherwise),
 *   dQ[j][:]          summed over the token range.
 * dH [T][N][d] is in the storage of V. */
int orc_route_all_bwd(const void *V, const void *K, const double *Q, const void *dH, double *dV,
                      double *dK, double *dQ, long long S, long long N, long long d, long long r,
                      long long first, long long T, int mode, int store, double eps, long long n0,
                      long long n1)
{
    struct orc_problem p = {V, K, Q, S, N, d, r, mode, store, eps};
    if (check_problem(&p, n0, n1) || Q == NULL || V == NULL || dH == NULL || dV == NULL ||
        dQ == NULL)
        return 1;
    if ((mode == ORC_KEYS_PROJECTED) != (dK != NULL))
        return 1;
    if (first < 1 || T < 1 || first + T - 1 > S)
        return 1;
    const long long nt = n1 - n0;
    const size_t esize = store == ORC_STORE_F32 ? 4 : store == ORC_STORE_BF16 ? 2 : 8;
    for (long long e = 0; e < S * nt * d; ++e)
        dV[e] = 0.0;
    if (dK)
        for (long long e = 0; e < S * nt * r; ++e)
            dK[e] = 0.0;
    const long long smax = first + T - 1;
    double *sdV = (double *)malloc(sizeof(double) * (size_t)(smax * nt * d));
    double *sdK = dK ? (double *)malloc(sizeof(double) * (size_t)(smax * nt * r)) : NULL;
    if (sdV == NULL || (dK != NULL && sdK == NULL)) {
        free(sdV);
        free(sdK);
        return 1;
    }
    int failed = 0;
    for (long long j = 0; j < T && !failed; ++j) {
        const long long sj = first + j;
        const void *dHj = (const char *)dH + (size_t)(j * N * d) * esize;
        if (orc_route_bwd(V, K, Q + j * r, dHj, sdV, sdK, dQ + j * r, sj, N, d, r, mode, store,
                          eps, n0, n1)) {
            failed = 1;
            break;
        }
        for (long long e = 0; e < sj * nt * d; ++e)
            dV[e] += sdV[e];
        if (dK)
            for (long long e = 0; e < sj * nt * r; ++e)
                dK[e] += sdK[e];
    }
    free(sdV);
    free(sdK);
    return failed;
}

/* The projected-key producer (Sec. 3.3, Eq. fused_projection): the output
 * projection of a residual-writing sub-layer and its key projection are one
 * matrix [W^O; W^K] with d + r rows, applied to the activation a_n that
 * enters the output projection:
 *   [o_n; k_n] = [W^O; W^K] a_n,   o_n in R^d (the residual value),
 *                                  k_n in R^r (its routing key).
 * A [N][m] holds a_n row by row; W [d + r][m] holds the rows of W^O then the
 * rows of W^K.  For tokens n in [n0, n1): O[n - n0][j] = sum_c W[j][c] A[n][c]
 * for j < d, and Kout[n - n0][j] = sum_c W[d + j][c] A[n][c] for j < r.  O may
 * be NULL when d = 0 (the embedding key of Eq. embedding_key_projection,
 * k_0 = W_0^K o_0, is this with d = 0 and a_n = o_0); Kout may be NULL when
 * r = 0 (a plain output projection). */
int orc_key_projection(const void *A, const void *W, double *O, double *Kout, long long N,
                       long long m, long long d, long long r, int store, long long n0,
                       long long n1)
{
    if (N < 0 || m < 1 || d < 0 || r < 0 || d + r < 1 || n0 < 0 || n1 < n0 || n1 > N)
        return 1;
    if (A == NULL || W == NULL || (d > 0 && O == NULL) || (r > 0 && Kout == NULL))
        return 1;
    if (store < 0 || store > 2)
        return 1;
#pragma omp parallel for schedule(static)
    for (long long n = n0; n < n1; ++n) {
        for (long long j = 0; j < d + r; ++j) {
            double acc = 0.0;
            for (long long c = 0; c < m; ++c)
                acc += widen(W, store, j * m + c) * widen(A, store, n * m + c);
            if (j < d)
                O[(n - n0) * d + j] = acc;
            else
                Kout[(n - n0) * r + (j - d)] = acc;
        }
    }
    return 0;
}

/* Backward of the projected-key producer [o_n; k_n] = [W^O; W^K] a_n
 * (Sec. 3.3, Eq. fused_projection).  The paper states no backward; for a
 * loss with upstream gradients g_n = [dO[n]; dK[n]] of the d + r outputs of
 * token n, the chain rule through the linear map C = A W^T gives
 *     dA[n][c] = sum_j g_n[j] W[j][c]        (j over the d + r outputs)
 *     dW[j][c] = sum_n g_n[j] A[n][c]        (n over the N tokens)
 * written out here as plain sums in fp64.  A [N][m], W [d + r][m], dO [N][d]
 * (NULL when d = 0), dK [N][r] (NULL when r = 0), all in storage `store`;
 * dA [N][m] and dW [d + r][m] are fp64.  Returns 0, or 1 on invalid input. */
int orc_key_projection_bwd(const void *A, const void *W, const void *dO, const void *dK,
                           double *dA, double *dW, long long N, long long m, long long d,
                           long long r, int store)
{
    if (N < 0 || m < 1 || d < 0 || r < 0 || d + r < 1 || store < 0 || store > 2)
        return 1;
    if (A == NULL || W == NULL || dA == NULL || dW == NULL || (d > 0 && dO == NULL) ||
        (r > 0 && dK == NULL))
        return 1;
    const long long nout = d + r;
#pragma omp parallel for schedule(static)
    for (long long n = 0; n < N; ++n) {
        for (long long c = 0; c < m; ++c) {
            double acc = 0.0;
            for (long long j = 0; j < nout; ++j) {
                const double g = j < d ? widen(dO, store, n * d + j) : widen(dK, store, n * r + (j - d));
                acc += g * widen(W, store, j * m + c);
            }
            dA[n * m + c] = acc;
        }
    }
#pragma omp parallel for schedule(static)
    for (long long j = 0; j < nout; ++j) {
        for (long long c = 0; c < m; ++c) {
            double acc = 0.0;
            for (long long n = 0; n < N; ++n) {
                const double g = j < d ? widen(dO, store, n * d + j) : widen(dK, store, n * r + (j - d));
                acc += g * widen(A, store, n * m + c);
            }
            dW[j * m + c] = acc;
        }
    }
    return 0;
}

/* Sets the number of OpenMP threads later parallel regions use (n >= 1);
 * no effect in a build without OpenMP.  Timing harness only. */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Number of OpenMP threads a parallel region of this library would use. */
int orc_num_threads(void)
{
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}
