// Host-side interface between the C ABI layer (argument validation) and the
// kernel launchers.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "lr_attnres.h"

namespace lrar {

struct Problem {
    const void *V;   // [S][N][d]
    const void *K;   // [S][N][r] (projected keys) or NULL
    const float *q;  // [r]
    int64_t S, N, d, r;
    int mode, dtype;
    float eps;
    int dh_dtype;    // storage of dH; differs from dtype only for block sources
};

// LRAR_OK if a kernel covers the (already validated) problem, else
// LRAR_EUNSUPPORTED with the reason in *why.  No HIP call.
int check_supported(const Problem &p, bool bwd, std::string *why);

// Workspace of the backward (per-workgroup dq partials).  No HIP call.
size_t bwd_workspace_bytes(const Problem &p);

int launch_fwd(const Problem &p, void *H, hipStream_t st, std::string *err);
// Online-softmax states of the sources in chunks of `chunk` (see
// lr_attnres_route_state_fwd): M, L [P][N], ACC [P][N][d] fp32.
int launch_state(const Problem &p, int64_t chunk, float *M, float *L, float *ACC, hipStream_t st,
                 std::string *err);
// H [N][d] (storage dtype) from P states (see lr_attnres_route_merge_fwd).
int launch_merge(const float *M, const float *L, const float *ACC, int64_t P, int64_t N, int64_t d,
                 int dtype, void *H, hipStream_t st, std::string *err);
// accumulate: add the gradients into dV, dK and dq instead of overwriting.
int launch_bwd(const Problem &p, const void *dH, void *dV, void *dK, float *dq, void *ws,
               bool accumulate, hipStream_t st, std::string *err);

// Largest dq-partial workspace the allocation-free backward serves from its
// file-scope device array (8 MiB per device).
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;

// launch_bwd (overwriting) with the dq partials in that device array instead
// of a caller workspace; LRAR_EUNSUPPORTED when the problem needs more.
// Allocates nothing; concurrent calls on one device race on the array.
int launch_bwd_noalloc(const Problem &p, const void *dH, void *dV, void *dK, float *dq,
                       hipStream_t st, std::string *err);

// One residual site of block-source routing (see lr_attnres_block_route_fwd).
struct BlockProblem {
    float *B;           // [nsrc][N][d] fp32 summary slots; slot nsrc-1 updated
    float *KB;          // [nsrc][N][r] fp32 key summaries (projected) or NULL
    const void *o_new;  // [N][d] newest sub-layer output, storage dtype
    const void *k_new;  // [N][r] its projected key, storage dtype, or NULL
    const float *q;     // [r]
    void *H;            // [N][d] storage dtype
    int64_t nsrc, N, d, r;
    int start, mode, dtype;
    float eps;
    // completed_bf16: the completed summaries are read from bf16 copies BC
    // [nsrc][N][d] (and KBC [nsrc][N][r], projected) instead of the fp32
    // slots (bf16 storage only), and `finish` writes slot nsrc-1's copy.
    int completed_bf16 = 0;
    void *BC = nullptr;
    void *KBC = nullptr;
    int finish = 0;
};

int check_block_supported(const BlockProblem &p, std::string *why);
int launch_block_fwd(const BlockProblem &p, hipStream_t st, std::string *err);

// The end of one site of the block reverse pass: the member o_new (and its
// projected key) leaves slot j (B[j] -= o_new, KB[j] -= k_new), and its
// gradient is the slot's gradient accumulated so far (dO = dB[j],
// dK = dKB[j], in the model dtype).
struct BlockRetire {
    float *B, *KB;
    const float *dB, *dKB;
    const void *o_new, *k_new;
    void *dO, *dK;
    int64_t j, N, d, r;
    int mode, dtype;
    bool grad_rows = false;  // dB / dKB are the slot's gradient rows themselves
};

hipError_t launch_block_retire(const BlockRetire &br, hipStream_t st);

// Phase 1 of the two-phase block inference (see lr_attnres_block_inter_fwd).
struct BlockInterProblem {
    const float *B, *KB;  // [nprev][N][d], [nprev][N][r] (projected) or NULL
    const float *Q;       // [nq][r]
    float *M, *L, *ACC;   // [nq][N], [nq][N], [nq][N][d]
    int64_t nprev, nq, N, d, r;
    int mode;
    float eps;
};

int launch_block_inter(const BlockInterProblem &p, hipStream_t st, std::string *err);

// Phase 2 at one site: p as for launch_block_fwd (p.nsrc - 1 = the partial
// slot); Ms, Ls, ACC this site's phase-1 state, or all NULL without one.
int launch_block_merge(const BlockProblem &p, const float *Ms, const float *Ls, const float *ACC,
                       hipStream_t st, std::string *err);

// One site of the block reverse pass: the routing backward over the fp32
// slots (p.dtype = F32, p.dh_dtype = the model dtype) accumulating into dB
// and dKB, dq written, then the retire step above.
int launch_block_bwd(const Problem &p, const BlockRetire &br, const void *dH, void *dB,
                     void *dKB, float *dq, void *ws, hipStream_t st, std::string *err);

// The deferred form of the same step (see lr_attnres_block_route_bwd_deferred):
// only the block in progress (the last slot) accumulates into the rows dP /
// dKP, the completed slots write their coefficients into coef
// [n_src - 1][3][N]; then the retire step with dB = dP, dKB = dKP.
int launch_block_bwd_deferred(const Problem &p, const BlockRetire &br, const void *dH, float *dP,
                              float *dKP, float *coef, float *dq, void *ws, hipStream_t st,
                              std::string *err);

// One site of the full-source deferred reverse pass (see
// lr_attnres_route_bwd_deferred): the coefficients of every source into
// coef [S][3][N] and dq; no gradient rows.
int launch_bwd_deferred_all(const Problem &p, const void *dH, float *coef, float *dq, void *ws,
                            hipStream_t st, std::string *err);

// A completed slot's gradient from the sites that read it as completed (see
// lr_attnres_block_gather_bwd).
struct BlockGather {
    const void *Bj, *KBj;   // the source's rows [N][d], key rows [N][r] or NULL (storage kdtype)
    const void *dHs;        // [n_sites][N][d] model dtype
    const float *Q;         // [n_sites][r]
    const float *coef;      // site u's coefficients at coef + u * site_stride ([3][N])
    int64_t site_stride, n_sites;
    void *dP, *dKP;         // [N][d], [N][r] or NULL, storage kdtype; overwritten
    int64_t N, d, r;
    int mode, dtype;
    float eps;
    // Storage of Bj, KBj, dP and dKP: fp32 for block summaries; the model
    // dtype for the sources of a full-source pass (lr_attnres_route_gather_bwd).
    int kdtype = LRAR_DTYPE_F32;
};

int check_gather_supported(const BlockGather &g, std::string *why);
int launch_block_gather(const BlockGather &g, hipStream_t st, std::string *err);

// Every read site of a pass over one source stack (see
// lr_attnres_route_all_fwd).
struct AllProblem {
    const void *V;    // [S][N][d]
    const void *K;    // [S][N][r] (projected keys) or NULL
    const float *Q;   // [T][r]
    void *H;          // [T][N][d]
    float *neff;      // [T][N] or NULL
    int64_t S, N, d, r, first, T;
    int mode, dtype;
    float eps;
};

int check_all_supported(const AllProblem &p, std::string *why);
// Whether the fused all-sites kernels take the problem (projected or sliced
// keys, S, T, r <= 64, d % 8 == 0); otherwise the sites run one by one.
bool all_fused(const AllProblem &p);
// The single-site problem of site j of an all-sites problem.
Problem all_site_problem(const AllProblem &p, int64_t j);

// Backward of every read site (see lr_attnres_route_all_bwd): dV [S][N][d],
// dK [S][N][r] (projected keys) or NULL, dQ [T][r]; overwritten, or added
// to when accumulating.  ws holds all_bwd_workspace_bytes(p) bytes.
size_t all_bwd_workspace_bytes(const AllProblem &p);
int check_all_bwd_supported(const AllProblem &p, std::string *why);
int launch_all_bwd(const AllProblem &p, const void *dH, void *dV, void *dK, float *dQ, void *ws,
                   bool accumulate, hipStream_t st, std::string *err);

// dq[j] (+)= sum_b partial[b][j] for j < ncols, in a fixed order.
hipError_t launch_dq_reduce(const float *partial, float *dq, int nblocks, int ncols,
                            bool accumulate, hipStream_t st);

// Effective number of sources of one site (see lr_attnres_route_neff); full
// rank is passed as sliced keys with r = d.
int launch_neff(const Problem &p, float *neff, hipStream_t st, std::string *err);

// The projected-key producer (see lr_attnres_key_proj_fwd).
struct KeyProjProblem {
    const void *A;  // [N][m]
    const void *W;  // [d + r][m]
    void *O;        // [N][d] or NULL
    void *K;        // [N][r] or NULL
    int64_t N, m, d, r;
    int dtype;
};

int check_key_proj_supported(const KeyProjProblem &p, std::string *why);
int launch_key_proj(const KeyProjProblem &p, hipStream_t st, std::string *err);
// Backward of the key producer: p.O and p.K are unused.  dW is fp32; the
// workspace holds the token splits' partials (key_proj_bwd_workspace_bytes).
void key_proj_bwd_splits(int64_t N, int64_t m, int64_t nout, int64_t *P, int64_t *per);
size_t key_proj_bwd_workspace_bytes(int64_t N, int64_t m, int64_t d, int64_t r);
int check_key_proj_bwd_supported(const KeyProjProblem &p, std::string *why);
int launch_key_proj_bwd(const KeyProjProblem &p, const void *dO, const void *dK, void *dA,
                        float *dW, void *workspace, hipStream_t st, std::string *err);
int launch_all_fwd(const AllProblem &p, hipStream_t st, std::string *err);

}  // namespace lrar
