/*
 * lr_attnres.h - C ABI of the MI355X (gfx950) depth-routing library of
 * Low-Rank Attention Residuals (LR-AttnRes), arXiv 2607.09694.
 *
 * At one residual read site every token n mixes its S cached sources
 * o_0..o_{S-1} (the embedding and the earlier sub-layer outputs, Sec. 3.1)
 * with softmax weights over depth computed from r-dimensional keys
 * (Sec. 3.2):
 *
 *     kbar_i  = RMSNorm(k_i),     rho_i = sqrt(mean_j k_ij^2 + eps),
 *                                  kbar_i = k_i / rho_i          (Eq. lr_key_norm)
 *     alpha_i = softmax_i(q^T kbar_i)                             (Eq. lr_attnres_weight)
 *     h       = sum_i alpha_i o_i                                 (Eq. lr_attnres_output)
 *
 * The RMSNorm has no gain (the paper's parameter-free convention, Appendix A
 * "Parameters"); eps is not given by the paper and is an explicit argument.
 * There is no score temperature.
 *
 * Key modes:
 *   LRAR_MODE_PROJECTED  k_i is row [i][n] of a separate key stack K[S][N][r]
 *                        (P-LR, Sec. 3.3, Eq. fused_projection).
 *   LRAR_MODE_SLICED     k_i = tail_r(o_i), the last r coordinates of the
 *                        value, read in place from V (S-LR, Sec. 3.4,
 *                        Eq. sliced_key); requires r <= d.
 *   LRAR_MODE_FULL       full-rank AttnRes: k_i = o_i, r must equal d
 *                        (Sec. 3.1, Eqs. attnres_weight / attnres_output).
 *
 * Layout: all arrays are dense and row-major.  V is [S][N][d] (source-major:
 * the rows of one source are contiguous, so the first S' sources of a deeper
 * stack are a valid S'-source stack), K and dK are [S][N][r], H and dH are
 * [N][d], q and dq are [r] fp32.  Sources are indexed in stack order,
 * i = 0 (embedding) .. S-1.  V, K, H, dH, dV, dK share one storage type,
 * fp32 or bf16; all arithmetic is fp32, and bf16 results are rounded to
 * nearest even.
 *
 * Ownership and execution: every pointer is caller-owned device memory.
 * The library allocates nothing, keeps no pointer after a call returns and
 * holds no state besides the per-thread error string.  Work is enqueued on
 * `stream` (a hipStream_t; NULL means the null stream) and runs
 * asynchronously: the caller keeps the buffers alive until the stream has
 * reached the work.  Results are bitwise reproducible from run to run.
 *
 * Errors: nothing is thrown across the ABI.  All arguments are validated on
 * the host before any HIP call, so an invalid call never touches the device:
 *   LRAR_EINVAL       a required pointer is NULL, a size is < 1 (N may be 0),
 *                     the mode or storage code is unknown, SLICED with r > d,
 *                     FULL with r != d, K or dK given outside PROJECTED,
 *                     eps negative or not finite, a tensor pointer not 16-byte
 *                     aligned (q and dq: 4-byte), an output overlapping an
 *                     input or another output, a size product overflowing
 *                     int64, or a workspace that is missing or too small.
 *   LRAR_EUNSUPPORTED a valid problem outside the kernels' limits (below).
 *   LRAR_EHIP         a HIP launch error; its text is in lr_attnres_last_error.
 * Limits: N <= 2^30; forward S <= 1024; backward S <= 512; backward of
 * PROJECTED/SLICED r <= 256; FULL, and every backward, d <= 4096 (bf16) or
 * d <= 2048 (fp32) when d is a multiple of 8 (bf16) or 4 (fp32), else
 * d <= 1024.
 */
#ifndef LR_ATTNRES_H
#define LR_ATTNRES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LR_ATTNRES_ABI_VERSION 1

enum { LRAR_MODE_PROJECTED = 0, LRAR_MODE_SLICED = 1, LRAR_MODE_FULL = 2 };
enum { LRAR_DTYPE_F32 = 0, LRAR_DTYPE_BF16 = 1 };
enum { LRAR_OK = 0, LRAR_EINVAL = 1, LRAR_EUNSUPPORTED = 2, LRAR_EHIP = 3 };

/*
 * Forward routing at one residual site (Sec. 3.2, Eqs. lr_key_norm,
 * lr_attnres_weight, lr_attnres_output; modes as above).
 *   V   [S][N][d]  values o_i, storage `dtype`, read only
 *   K   [S][N][r]  keys, storage `dtype`; PROJECTED only, else must be NULL
 *   q   [r]        fp32 pseudo-query of this site
 *   H   [N][d]     output h, storage `dtype`, fully overwritten
 * The softmax weights are not stored.  Returns LRAR_OK or an error code.
 */
int lr_attnres_route_fwd(const void *V, const void *K, const float *q, void *H,
                         int64_t S, int64_t N, int64_t d, int64_t r,
                         int mode, int dtype, float eps, void *stream);

/*
 * Bytes of device workspace lr_attnres_route_bwd needs for this problem
 * (per-workgroup partial sums of dq).  0 for an invalid problem.
 */
size_t lr_attnres_route_bwd_workspace_bytes(int64_t S, int64_t N, int64_t d, int64_t r,
                                            int mode, int dtype);

/*
 * Backward of the forward above for the loss L = sum_n dH[n] . h[n].  The
 * paper gives no backward; this is the gradient of its Eqs. lr_key_norm,
 * lr_attnres_weight and lr_attnres_output (the weights are recomputed from
 * the keys, not saved, as Appendix A "Activation memory" assumes):
 *     g_i  = dH . o_i,   ds_i = alpha_i (g_i - sum_l alpha_l g_l)
 *     dV_i = alpha_i dH  (+ the key path below for SLICED and FULL)
 *     dk_i = (ds_i / rho_i) (q - kbar_i s_i / r),   s_i = q . kbar_i
 *     dq   = sum_n sum_i ds_i kbar_i
 *   V, K, q      as in the forward, read only
 *   dH  [N][d]   upstream gradient, storage `dtype`, read only
 *   dV  [S][N][d] storage `dtype`, fully overwritten.  SLICED adds dk_i into
 *                the last r coordinates, FULL into all d coordinates.
 *   dK  [S][N][r] storage `dtype`, PROJECTED only (fully overwritten), else NULL
 *   dq  [r]      fp32, overwritten with the sum over all N tokens (0 if N = 0);
 *                the sum is taken in a fixed order, so it is reproducible.
 *   workspace    device scratch of at least
 *                lr_attnres_route_bwd_workspace_bytes(...) bytes (16-byte
 *                aligned; may be NULL when that size is 0).  Its contents on
 *                entry are ignored; it must not overlap any other argument,
 *                and two calls in flight must not share it.
 */
int lr_attnres_route_bwd(const void *V, const void *K, const float *q, const void *dH,
                         void *dV, void *dK, float *dq, void *workspace,
                         size_t workspace_bytes, int64_t S, int64_t N, int64_t d, int64_t r,
                         int mode, int dtype, float eps, void *stream);

/*
 * The same backward, accumulating: dV += (its gradient), dK += (projected
 * keys), dq += (sum over tokens), instead of overwriting them.  This is the
 * form a model pass needs: each cached source o_i receives gradient from
 * every later residual site (Sec. 3.1: site t reads all sources written
 * before it), so the caller keeps one dV stack and adds each site's
 * contribution in place, saving a separate read-add-write pass over it.
 * Arguments, validation and errors are those of lr_attnres_route_bwd; the
 * gradient buffers must hold valid values on entry (zeros to start).
 */
int lr_attnres_route_bwd_accumulate(const void *V, const void *K, const float *q,
                                    const void *dH, void *dV, void *dK, float *dq,
                                    void *workspace, size_t workspace_bytes, int64_t S,
                                    int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                    float eps, void *stream);

/*
 * lr_attnres_route_bwd without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  The per-workgroup dq partials go to a
 * device array that the library holds, 8 MiB on every device it runs on,
 * kept until the process ends (its address is looked up once per device, on
 * that device's first call).  The call itself allocates nothing, on the
 * device or through any library routine.
 *   Arguments, results, validation and errors are those of
 *   lr_attnres_route_bwd with the workspace removed, plus LRAR_EUNSUPPORTED
 *   when the problem needs more than 8 MiB of partials
 *   (lr_attnres_route_bwd_workspace_bytes > 8388608: e.g. r = 32 beyond
 *   2^19 tokens with projected keys, or full rank at d = 1024 beyond
 *   32768 tokens).
 *   All calls on one device share the array, and each call leaves its
 *   partials there: two calls that can run at the same time on one device
 *   (different streams, or different host threads without ordering) race
 *   and may return wrong dq.  Calls ordered on one stream are safe; nothing
 *   in the array needs to start at zero.
 */
int lr_attnres_route_bwd_noalloc(const void *V, const void *K, const float *q,
                                 const void *dH, void *dV, void *dK, float *dq, int64_t S,
                                 int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                 float eps, void *stream);

/*
 * Block-source routing forward at one residual site: Block AttnRes (Sec. 3.1,
 * Eqs. block_attnres_sum and block_attnres_partial_sum) with the low-rank
 * keys of Sec. 3.2.  The 2L sub-layer outputs are grouped into consecutive
 * blocks; site t reads the embedding, every completed block summary and the
 * partial summary of the block in progress.  The summaries are kept by the
 * caller in fp32 slots, updated here one member at a time:
 *   B   [n_src][N][d] fp32  slot 0 = embedding, slot j >= 1 = sum of block j's
 *                           outputs so far.  Slot n_src-1 is updated in place:
 *                           B[n_src-1] = (start ? 0 : B[n_src-1]) + o_new.
 *   KB  [n_src][N][r] fp32  projected keys only (else NULL): the key of a
 *                           summary is the sum of its members' keys, updated
 *                           like B with k_new.  Sliced keys are the last r
 *                           columns of each slot (the tail of the summed row).
 *   o_new [N][d], k_new [N][r]  the newest sub-layer output and its projected
 *                           key (k_new NULL for sliced keys), storage `dtype`.
 *   q [r] fp32; H [N][d] storage `dtype`, fully overwritten.
 * The routing over slots 0..n_src-1 (after the update) is that of
 * lr_attnres_route_fwd.  A model pass calls this once per site: at site 1
 * with o_new = the embedding, n_src = 1, start = 1; at site t >= 2 with
 * o_new = o_{t-1}, which belongs to block j = floor((t-2)/c) + 1 for blocks
 * of c outputs, so n_src = j + 1 and start = ((t-2) mod c == 0).
 * The reading that a summary's key is the sum of its members' keys is this
 * library's (the paper does not define block keys for projected keys).
 * Full-rank keys (block AttnRes itself, r = d) run as sliced keys over the
 * whole row, which Sec. 3.4 states is the same routing.
 * Errors as for lr_attnres_route_fwd, plus EINVAL for start not 0/1 and for
 * an unknown mode; d not a multiple of 4, d > 2048 and n_src > 1024 are
 * EUNSUPPORTED.  k_new needs only element alignment (it is
 * read element by element), the other tensors 16 bytes.  H must not overlap
 * any other argument; B and KB are rewritten and must not overlap the inputs.
 */
int lr_attnres_block_route_fwd(float *B, float *KB, const void *o_new, const void *k_new,
                               const float *q, void *H, int64_t n_src, int start, int64_t N,
                               int64_t d, int64_t r, int mode, int dtype, float eps,
                               void *stream);

/*
 * The same site with the completed block summaries stored in bf16 (bf16
 * storage only).  Block AttnRes (Sec. 3.1) reads every completed summary at
 * every later site; this keeps them as bf16 copies, which halves those
 * reads.  The paper states no precision for the summaries; this storage
 * option is the library's reading:
 *   - slot n_src-1 (the one o_new joins) is updated in the fp32 B / KB
 *     exactly as in lr_attnres_block_route_fwd and routed from fp32;
 *   - slots 0..n_src-2 (completed) are read from BC [.][N][d] bf16 and, for
 *     projected keys, KBC [.][N][r] bf16, instead of B and KB;
 *   - finish = 1 (o_new is the last member of its block, or the embedding)
 *     also writes BC[n_src-1] (and KBC[n_src-1]): the updated fp32 row
 *     rounded once to bf16, round to nearest even.
 * A model pass sets finish at site 1 (the embedding) and at every site
 * whose o_new completes a block of c, t - 1 = jc, so each copy is the fp32
 * member-order sum of its block, rounded once.
 * BC / KBC need 16-byte alignment.  BC is required when N > 0 and either
 * n_src > 1 or finish = 1; KBC likewise with projected keys, NULL
 * otherwise.  Errors and limits as for lr_attnres_block_route_fwd, plus
 * EINVAL for finish not 0/1; BC and KBC must not overlap any other
 * argument.
 */
int lr_attnres_block_route_fwd_bf16c(float *B, float *KB, void *BC, void *KBC,
                                     const void *o_new, const void *k_new, const float *q,
                                     void *H, int64_t n_src, int start, int finish, int64_t N,
                                     int64_t d, int64_t r, int mode, float eps, void *stream);

/*
 * Block-source backward at one residual site, for the reverse pass of a
 * model that ran lr_attnres_block_route_fwd at every site (Sec. 3.1 "Block
 * AttnRes" with Sec. 3.2; the gradient of L = sum_n dH[n] . h[n]).  Sites are
 * visited in reverse order.  On entry the slots hold what the forward of this
 * site saw (slot n_src-1 includes o_new); on return:
 *   dB  [n_src][N][d] fp32 += the gradient of each slot (value path and, for
 *                       sliced keys, the key path in the last r columns);
 *   dKB [n_src][N][r] fp32 += the gradient of each key summary (projected;
 *                       else NULL);
 *   dO  [N][d], dK [N][r] (storage `dtype`) = dB[n_src-1], dKB[n_src-1]: a
 *                       summary is the plain sum of its members, so the member
 *                       o_new receives its slot's gradient, which at this
 *                       point holds the contributions of every later site;
 *   B[n_src-1] -= o_new, KB[n_src-1] -= k_new: the member leaves its slot, so
 *                       the previous site sees its own partial summary;
 *   dq [r] fp32 = this site's query gradient (summed over tokens).
 *   dH [N][d] is in storage `dtype`; workspace as for lr_attnres_route_bwd
 *   with S = n_src, LRAR_DTYPE_F32 and, for full-rank keys, LRAR_MODE_SLICED.
 * Limits: those of lr_attnres_block_route_fwd and of the backward (so
 * full-rank keys, which run as sliced keys with r = d, need d <= 256).  Outputs
 * (B, KB, dB, dKB, dO, dK, dq, workspace) must not overlap each other or the
 * inputs (o_new, k_new, q, dH).  Removing o_new from the fp32 slot by
 * subtraction differs from the forward's partial sum by fp32 rounding only.
 */
int lr_attnres_block_route_bwd(float *B, float *KB, float *dB, float *dKB, const void *o_new,
                               const void *k_new, const float *q, const void *dH, void *dO,
                               void *dK, float *dq, void *workspace, size_t workspace_bytes,
                               int64_t n_src, int64_t N, int64_t d, int64_t r, int mode,
                               int dtype, float eps, void *stream);

/*
 * The block reverse pass in deferred form: the same gradients as
 * lr_attnres_block_route_bwd, with the fp32 gradient of a completed slot
 * formed once instead of read-modified-written at every later site.  A
 * completed slot j is read by every site after its block completes; at such
 * a site t its gradient is alpha_{t,j} dH_t plus, on the key, the RMSNorm
 * term (ds/rho) q_t - (ds s/(rho r)) kbar_j, so the site only records three
 * numbers per token, and lr_attnres_block_gather_bwd later sums them.  The
 * block in progress (slot n_src - 1) keeps a running gradient.
 *
 * One site (arguments as for lr_attnres_block_route_bwd, except):
 *   dP  [N][d] fp32: the running gradient of the block in progress, += this
 *       site's contribution (value path and, for sliced keys, the key path
 *       in the last r columns); dKP [N][r] fp32 likewise for projected keys;
 *   coef [n_src - 1][3][N] fp32, overwritten: for each completed slot i,
 *       alpha_i, ds_i / rho_i and ds_i s_i / (rho_i r) per token (NULL when
 *       n_src = 1);
 *   dO = dP, dK = dKP (model dtype) after the addition; B[n_src - 1] -= o_new,
 *   KB[n_src - 1] -= k_new; dq [r] = this site's query gradient.
 * Driving a model pass in reverse: when slot j first becomes the block in
 * progress (the last site of block j), set dP, dKP with
 * lr_attnres_block_gather_bwd over the sites that read slot j as completed
 * (zero sites: zeros), then call this function at each site down to the
 * block's first.  Limits and errors as for lr_attnres_block_route_bwd.
 */
int lr_attnres_block_route_bwd_deferred(float *B, float *KB, float *dP, float *dKP, float *coef,
                                        const void *o_new, const void *k_new, const float *q,
                                        const void *dH, void *dO, void *dK, float *dq,
                                        void *workspace, size_t workspace_bytes, int64_t n_src,
                                        int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                        float eps, void *stream);

/*
 * The gradient of completed slot `slot` from the n_sites sites that read it
 * as completed (see lr_attnres_block_route_bwd_deferred):
 *   dP [N][d] = sum_u alpha_u dH_u  + (key columns) sum_u cq_u q_u - (sum_u ck_u) kbar
 *   (sliced keys: the last r columns; projected keys: dKP [N][r] takes the
 *   key term and dP the value term), overwritten.
 *   B [.][N][d], KB [.][N][r] fp32: the slots; the slot's key kbar = k / rho
 *   is recomputed from B[slot] (sliced) or KB[slot] (projected);
 *   dHs [n_sites][N][d] model dtype: the sites' dH, in site order;
 *   Q [n_sites][r] fp32: their queries;
 *   coef: site u's coefficients (alpha, cq, ck) for this slot are the three
 *   [N] rows at coef + u * coef_site_stride (floats; >= 3 N).
 * EUNSUPPORTED: d not a multiple of 4 or above 2048, more than 1024 sites,
 * n_sites * r above 16384.  Other errors as for lr_attnres_block_route_bwd.
 */
int lr_attnres_block_gather_bwd(const float *B, const float *KB, int64_t slot, const void *dHs,
                                const float *Q, const float *coef, int64_t coef_site_stride,
                                int64_t n_sites, float *dP, float *dKP, int64_t N, int64_t d,
                                int64_t r, int mode, int dtype, float eps, void *stream);

/*
 * Split-sources forward (Sec. 3.5's merge of online-softmax states, applied
 * to the sources of one site): the S sources are cut into P = ceil(S / chunk)
 * consecutive chunks, and chunk p's state over sources p chunk ..
 * min(S, (p + 1) chunk) - 1 is written per token:
 *   M [P][N] = max score, L [P][N] = sum exp(s - M),
 *   ACC [P][N][d] = sum exp(s - M) o_i      (all fp32, overwritten),
 * with the scores of lr_attnres_route_fwd (same V, K, q, mode, dtype, eps).
 * ACC / L is the routing over that chunk alone.  The states are what a pass
 * whose sources are spread over several devices would exchange, and they
 * route a stack deeper than one call takes (S above 1024);
 * lr_attnres_route_merge_fwd turns them into h.  (For few tokens on one
 * device, lr_attnres_route_fwd already splits each token's sources over a
 * workgroup and merges in on-chip memory, which is faster than states plus
 * a merge.)  M and L need 4-byte alignment, ACC 16 bytes; V, K and q as for
 * lr_attnres_route_fwd.
 * EINVAL: chunk < 1, or as lr_attnres_route_fwd.  EUNSUPPORTED: chunk above
 * 1024, more than 65535 chunks, or the row limits of lr_attnres_route_fwd.
 */
int lr_attnres_route_state_fwd(const void *V, const void *K, const float *q, float *M, float *L,
                               float *ACC, int64_t S, int64_t N, int64_t d, int64_t r,
                               int64_t chunk, int mode, int dtype, float eps, void *stream);

/*
 * H [N][d] (storage `dtype`) = sum_p e^(M_p - m) ACC_p / sum_p e^(M_p - m) L_p,
 * m = max_p M_p: the routing over the union of the P chunks whose states
 * (layout of lr_attnres_route_state_fwd) are given; with the states of all
 * chunks of one site it equals lr_attnres_route_fwd's h up to rounding.
 * M and L need 4-byte alignment, ACC and H 16 bytes.
 * EINVAL: P < 1, N < 0, d < 1, unknown dtype, misaligned or overlapping
 * buffers.  EUNSUPPORTED: P above 1024 or N above 2^30 (any row width:
 * wide rows are split into column blocks).
 */
int lr_attnres_route_merge_fwd(const float *M, const float *L, const float *ACC, void *H,
                               int64_t P, int64_t N, int64_t d, int dtype, void *stream);

/*
 * Two-phase block inference (Sec. 3.5): the site queries do not depend on
 * the input, and routing over the completed slots merges with routing over
 * the partial block by an online-softmax update.  The c sites whose newest
 * output falls in one block all read the same completed slots 0..n_prev-1,
 * so phase 1 reads those slot rows once for all of their queries:
 *   B [n_prev][N][d] fp32, KB [n_prev][N][r] fp32 (projected, else NULL):
 *     the completed slots, as in lr_attnres_block_route_fwd;
 *   Q [n_queries][r] fp32: the queries of those sites;
 *   M, L [n_queries][N] fp32, ACC [n_queries][N][d] fp32, overwritten with
 *     each query's state: M = max score, L = sum exp(s - M),
 *     ACC = sum exp(s - M) b_i  (so ACC / L is the routing over those slots).
 * EUNSUPPORTED beyond 1024 completed slots or 64 queries, or d not a
 * multiple of 4.
 */
int lr_attnres_block_inter_fwd(const float *B, const float *KB, const float *Q, float *M,
                               float *L, float *ACC, int64_t n_prev, int64_t n_queries,
                               int64_t N, int64_t d, int64_t r, int mode, float eps,
                               void *stream);

/*
 * Phase 2 at one site: slot `slot` (the block in progress, = n_prev) gains
 * o_new exactly as in lr_attnres_block_route_fwd with n_src = slot + 1, and
 * its score merges into the site's phase-1 state (M, L: [N], ACC: [N][d], the
 * rows of this site's query; all NULL when slot = 0, where there are no
 * completed slots):
 *   m' = max(M, s), h = (e^(M-m') ACC + e^(s-m') b_slot) / (e^(M-m') L + e^(s-m')).
 * H [N][d] in storage `dtype` equals lr_attnres_block_route_fwd's h up to
 * rounding.  Errors and limits as for lr_attnres_block_route_fwd.
 */
int lr_attnres_block_merge_fwd(float *B, float *KB, const void *o_new, const void *k_new,
                               const float *q, const float *M, const float *L, const float *ACC,
                               void *H, int64_t slot, int start, int64_t N, int64_t d, int64_t r,
                               int mode, int dtype, float eps, void *stream);

/*
 * The reverse pass of a full-source model in deferred form (gradient of
 * Sec. 3.1 Eq. full_attnres_source_set with Sec. 3.2; the paper states no
 * backward).  Site t reads the sources 0 .. t-1 and is the only site that
 * has source t-1 as its newest; once site t's backward is done, every site
 * that reads source t-1 has recorded its share, so source t-1's gradient is
 * final.  Instead of adding into the gradient rows of all t sources at every
 * site (lr_attnres_route_bwd_accumulate), each site records three numbers
 * per source and token, and one gather per source then forms that source's
 * whole gradient from the sites that read it: dV_i = sum_t alpha_{t,i} dH_t
 * plus, on the key, sum_t (ds/rho) q_t - (sum_t ds s/(rho r)) kbar_i.
 *
 * lr_attnres_route_bwd_deferred: one site, arguments as for
 * lr_attnres_route_bwd except that no gradient rows are written:
 *   coef [S][3][N] fp32, overwritten: for every source i of the site,
 *        alpha_i, ds_i / rho_i and ds_i s_i / (rho_i r) per token;
 *   dq [r] fp32: the site's query gradient (summed over tokens).
 * Projected or sliced keys (full-rank keys: EUNSUPPORTED); other limits and
 * errors as for lr_attnres_route_bwd, with coef among the outputs.
 *
 * lr_attnres_route_gather_bwd: the gradient of one source from the n_sites
 * sites that read it:
 *   V [S][N][d], K [S][N][r] (projected, else NULL): the stacks; only plane
 *        `source` is read (its key: the last r columns of V or K's row);
 *   dHs [n_sites][N][d] storage `dtype`, Q [n_sites][r] fp32: those sites'
 *        upstream gradients and queries, in the order of their coefficients;
 *   coef: site u's coefficients for this source at coef + u * coef_site_stride
 *        (3 rows of N floats, as written by lr_attnres_route_bwd_deferred at
 *        that site plus 3 N * source); coef_site_stride >= 3 N;
 *   dV [N][d], dK [N][r] (projected, else NULL) storage `dtype`, overwritten:
 *        the source's gradient (with sliced keys the key path is in the last
 *        r columns of dV).  n_sites = 0 writes zeros.
 * EINVAL for source outside [0, S), negative n_sites, a short stride,
 * misalignment (V, dV, dHs 16 bytes) or overlap of the outputs with the
 * inputs; EUNSUPPORTED for full-rank keys, d % 4 != 0 or d > 2048,
 * n_sites > 1024 or n_sites * r > 16384, N > 2^30.
 * Driving the reverse pass: for t = T down to 1, lr_attnres_route_bwd_deferred
 * at site t, then lr_attnres_route_gather_bwd for source t - 1 over sites
 * t .. T.  The results equal the accumulating pass up to rounding order.
 */
int lr_attnres_route_bwd_deferred(const void *V, const void *K, const float *q, const void *dH,
                                  float *coef, float *dq, void *workspace, size_t workspace_bytes,
                                  int64_t S, int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                  float eps, void *stream);
int lr_attnres_route_gather_bwd(const void *V, const void *K, int64_t source, const void *dHs,
                                const float *Q, const float *coef, int64_t coef_site_stride,
                                int64_t n_sites, void *dV, void *dK, int64_t S, int64_t N,
                                int64_t d, int64_t r, int mode, int dtype, float eps,
                                void *stream);

/*
 * Every read site of a pass over one stack of sources, in one call (Sec. 3.1,
 * Eq. full_attnres_source_set: site t reads the sources 0 .. t-1; routing of
 * Sec. 3.2 with any of the three key modes, Sec. 3.3-3.4), with each site's
 * effective number of sources (Sec. 4.5, Eq. effective_sources).  For use once
 * all outputs of the pass exist: recomputing the routed states of a pass,
 * probing a trained model.  Site j = 0 .. T-1 reads the first `first + j`
 * sources:
 *   V    [S][N][d] storage `dtype`: the sources o_0 .. o_{S-1};
 *   K    [S][N][r] storage `dtype`: their projected keys, or NULL for sliced
 *        keys (the last r columns of V);
 *   Q    [T][r] fp32: the sites' queries, row j for site j;
 *   H    [T][N][d] storage `dtype`, overwritten: row (j, n) is site j's
 *        routed state of token n (as lr_attnres_route_fwd over the first
 *        first + j sources with query Q[j]);
 *   neff [T][N] fp32, overwritten, or NULL: exp(-sum_i alpha_i log alpha_i)
 *        of site j's weights for token n.
 * With projected or sliced keys, S, T and r at most 64 and d a multiple of
 * 8, one fused launch reads the stack once for all sites; otherwise (full-rank
 * keys, larger S, T or r, other d) the library runs the sites one after the
 * other, each as lr_attnres_route_fwd over its prefix (and
 * lr_attnres_route_neff), so every site's H row is bit for bit that call's.
 * EINVAL: first < 1, T < 1, first + T - 1 > S, or the conditions of
 * lr_attnres_route_fwd (V, H 16-byte aligned; K, Q, neff element aligned; no
 * output may overlap an input or the other output).  EUNSUPPORTED: N above
 * 2^30, or, site by site, what lr_attnres_route_fwd refuses for the last site
 * (first + T - 1 sources).  In the fused launch non-finite source values are
 * not confined to the sites that read them: a source past a site's prefix
 * enters that site's product with weight 0, and 0 * inf is NaN.
 */
int lr_attnres_route_all_fwd(const void *V, const void *K, const float *Q, void *H, float *neff,
                             int64_t S, int64_t N, int64_t d, int64_t r, int64_t first,
                             int64_t T, int mode, int dtype, float eps, void *stream);

/*
 * Backward of every read site of a pass (the gradient of
 * lr_attnres_route_all_fwd; the paper states no backward).  For the loss
 * L = sum_j sum_n dH[j][n] . h_j[n], with the sites, V, K, Q and the limits
 * of lr_attnres_route_all_fwd:
 *   dH [T][N][d] storage `dtype`: row (j, n) is dL/dh_j[n];
 *   dV [S][N][d] storage `dtype`: dL/dV, the sum over the sites that read
 *        each source (zero rows for sources no site reads); with sliced keys
 *        it includes the key path through the last r columns;
 *   dK [S][N][r] storage `dtype`: dL/dK with projected keys, else NULL;
 *   dQ [T][r] fp32: row j is dL/dQ[j], summed over the N tokens;
 *   workspace: lr_attnres_route_all_bwd_workspace_bytes(...) bytes of device
 *        memory, 4-byte aligned (per-workgroup dQ partials).
 * accumulate = 0 overwrites dV, dK and dQ; 1 adds the gradients to them.
 * Where the fused forward applies and storage is bf16, one fused launch moves
 * each source row, upstream row and dV row once for all sites and rounds each
 * gradient to bf16 once.  Otherwise (full-rank keys, fp32 storage, larger S,
 * T or r, other d) the sites run one after the other as accumulating
 * lr_attnres_route_bwd calls over their prefixes, after a fill kernel has
 * zeroed dV, dK and dQ when overwriting (no memset); a source's gradient is
 * then rounded to the storage after each site that reads it, and dQ row j is
 * bit for bit site j's dq.  Either way dQ is reduced in a fixed order, so
 * results are bitwise reproducible.
 * EINVAL as for lr_attnres_route_all_fwd, plus dH, dV 16-byte aligned, dK and
 * dQ element aligned, a too small workspace, accumulate not 0 or 1, and any
 * output (or the workspace) overlapping an input or another output.
 * EUNSUPPORTED: N above 2^30, or, site by site, what lr_attnres_route_bwd
 * refuses for the last site.  The workspace query covers whichever path the
 * problem takes (the single-site backward's workspace when site by site).
 */
size_t lr_attnres_route_all_bwd_workspace_bytes(int64_t S, int64_t N, int64_t d, int64_t r,
                                                int64_t first, int64_t T, int mode, int dtype);
int lr_attnres_route_all_bwd(const void *V, const void *K, const float *Q, const void *dH,
                             void *dV, void *dK, float *dQ, void *workspace,
                             size_t workspace_bytes, int64_t S, int64_t N, int64_t d, int64_t r,
                             int64_t first, int64_t T, int mode, int dtype, float eps,
                             int accumulate, void *stream);

/*
 * Effective number of sources of one read site (Sec. 4.5, Eq.
 * effective_sources): neff[n] = exp(-sum_i alpha_i log alpha_i) of token n's
 * routing weights (Eq. lr_attnres_weight) over the S sources.  Reads the
 * keys only.  Arguments and errors as for lr_attnres_route_fwd, with neff
 * [N] fp32 (4-byte aligned) in place of H; V may be NULL with projected
 * keys.  EUNSUPPORTED above S = 1024 or N = 2^30.
 */
int lr_attnres_route_neff(const void *V, const void *K, const float *q, float *neff, int64_t S,
                          int64_t N, int64_t d, int64_t r, int mode, int dtype, float eps,
                          void *stream);

/*
 * The projected-key producer (Sec. 3.3, Eq. fused_projection): the output
 * projection W^O [d][m] of a residual-writing sub-layer and its key
 * projection W^K [r][m] stacked as one matrix, applied to the activations
 * entering the output projection, so that each sub-layer emits its residual
 * value and its routing key in one pass:
 *   A [N][m]     storage `dtype`: row n is a_n (the attention output before
 *                its output projection, or the gated SwiGLU hidden state);
 *   W [d + r][m] storage `dtype`: rows 0 .. d-1 are W^O, rows d .. d+r-1 are
 *                W^K (the [out][in] layout of a linear layer's weight);
 *   O [N][d]     overwritten with o_n = W^O a_n, rounded to nearest even:
 *                typically the sub-layer's plane V + i*N*d of the value stack;
 *   K [N][r]     overwritten with k_n = W^K a_n: typically K + i*N*r.
 * d = 0 (O NULL) gives a key projection alone, e.g. the embedding key
 * k_0 = W_0^K o_0 of Eq. embedding_key_projection; r = 0 (K NULL) a plain
 * output projection.  fp32 accumulation.  EINVAL: N < 0, m < 1, d or r < 0,
 * d + r < 1, A or W NULL or not 16-byte aligned (N > 0), O (K) NULL with
 * d > 0 (r > 0) or non-NULL with d = 0 (r = 0), O or K not element aligned,
 * outputs overlapping each other or the inputs.  EUNSUPPORTED: fp32 storage,
 * m % 8 != 0, m or d + r above 2^20, N above 2^30.
 */
int lr_attnres_key_proj_fwd(const void *A, const void *W, void *O, void *K, int64_t N, int64_t m,
                            int64_t d, int64_t r, int dtype, void *stream);

/* Backward of the projected-key producer (Sec. 3.3, Eq. fused_projection).
 * The paper gives no backward; with upstream gradients G = [dO, dK] of the
 * d value and r key outputs of each token, the chain rule through
 * [o_n; k_n] = [W^O; W^K] a_n gives
 *   dA [N][m]     = dO W^O + dK W^K, storage `dtype`, rounded to nearest
 *                   even from fp32 sums over the d + r outputs;
 *   dW [d + r][m] = [dO^T A; dK^T A], fp32 (overwritten, not accumulated),
 *                   fp32 sums over the N tokens, in a fixed order (bitwise
 *                   reproducible); N = 0 gives dW = 0.
 * A [N][m] and W [d + r][m] are the forward's inputs, dO [N][d] (NULL when
 * d = 0) and dK [N][r] (NULL when r = 0) the upstream gradients, all in
 * storage `dtype`.  `workspace` is caller-owned device memory of at least
 * lr_attnres_key_proj_bwd_workspace_bytes(N, m, d, r, dtype) bytes (the
 * fp32 partials of dW when its token sum is split; may be NULL when that
 * is 0); its contents on entry do not matter.  Asynchronous on `stream`.
 * EINVAL: N < 0, m < 1, d or r < 0, d + r < 1, a required pointer NULL or
 * not 16-byte aligned, dO (dK) non-NULL with d = 0 (r = 0), the workspace
 * too small, outputs (dA, dW, workspace) overlapping each other or the
 * inputs.  EUNSUPPORTED: fp32 storage, m, d or r not a multiple of 8, m or
 * d + r above 2^20, N above 2^30.
 */
size_t lr_attnres_key_proj_bwd_workspace_bytes(int64_t N, int64_t m, int64_t d, int64_t r,
                                               int dtype);
int lr_attnres_key_proj_bwd(const void *A, const void *W, const void *dO, const void *dK,
                            void *dA, float *dW, void *workspace, size_t workspace_bytes,
                            int64_t N, int64_t m, int64_t d, int64_t r, int dtype, void *stream);

/* Text of the last error raised on the calling thread ("" if none); valid
 * until the next call into the library on that thread. */
const char *lr_attnres_last_error(void);

/* LR_ATTNRES_ABI_VERSION of the built library. */
int lr_attnres_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LR_ATTNRES_H */
