// C ABI entry points of the routing library: argument validation (entirely
// on the host, before any HIP call) and dispatch to the kernel launchers.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <string>

#include "lr_attnres.h"
#include "route_launch.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string &msg)
{
    g_last_error = msg;
    return code;
}

bool mul_ok(int64_t a, int64_t b, int64_t *out) { return !__builtin_mul_overflow(a, b, out); }

struct Span {
    const char *name;
    uintptr_t lo, hi;  // [lo, hi)
};

Span span(const char *name, const void *p, int64_t bytes)
{
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{name, lo, p ? lo + (uintptr_t)bytes : lo};
}

bool overlaps(const Span &a, const Span &b)
{
    return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}

// Shapes, mode, storage, eps.  Fills the element counts on success.
int check_shape(int64_t S, int64_t N, int64_t d, int64_t r, int mode, int dtype, float eps,
                int64_t *v_elems, int64_t *k_elems, int64_t *h_elems)
{
    if (mode != LRAR_MODE_PROJECTED && mode != LRAR_MODE_SLICED && mode != LRAR_MODE_FULL)
        return fail(LRAR_EINVAL, "unknown key mode " + std::to_string(mode));
    if (dtype != LRAR_DTYPE_F32 && dtype != LRAR_DTYPE_BF16)
        return fail(LRAR_EINVAL, "unknown storage type " + std::to_string(dtype));
    if (S < 1 || d < 1 || r < 1 || N < 0)
        return fail(LRAR_EINVAL, "sizes must satisfy S >= 1, N >= 0, d >= 1, r >= 1");
    if (mode == LRAR_MODE_SLICED && r > d)
        return fail(LRAR_EINVAL, "sliced keys need r <= d");
    if (mode == LRAR_MODE_FULL && r != d)
        return fail(LRAR_EINVAL, "full-rank keys need r == d");
    if (!isfinite(eps) || eps < 0.0f)
        return fail(LRAR_EINVAL, "eps must be finite and >= 0");
    const int64_t esize = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t sn, vb, kb, hb;
    if (!mul_ok(S, N, &sn) || !mul_ok(sn, d, v_elems) || !mul_ok(*v_elems, esize, &vb) ||
        !mul_ok(sn, r, k_elems) || !mul_ok(*k_elems, esize, &kb) || !mul_ok(N, d, h_elems) ||
        !mul_ok(*h_elems, esize, &hb))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    return LRAR_OK;
}

int check_ptr(const void *p, const char *name, size_t align, bool required)
{
    if (!p) {
        if (required)
            return fail(LRAR_EINVAL, std::string(name) + " is NULL");
        return LRAR_OK;
    }
    if (reinterpret_cast<uintptr_t>(p) % align != 0)
        return fail(LRAR_EINVAL, std::string(name) + " is not " + std::to_string(align) +
                                     "-byte aligned");
    return LRAR_OK;
}

// No output may overlap an input or another output.
int check_aliasing(const Span *outs, int nout, const Span *ins, int nin)
{
    for (int a = 0; a < nout; ++a) {
        for (int b = 0; b < nin; ++b)
            if (overlaps(outs[a], ins[b]))
                return fail(LRAR_EINVAL, std::string("output ") + outs[a].name +
                                             " overlaps input " + ins[b].name);
        for (int b = a + 1; b < nout; ++b)
            if (overlaps(outs[a], outs[b]))
                return fail(LRAR_EINVAL, std::string("outputs ") + outs[a].name + " and " +
                                             outs[b].name + " overlap");
    }
    return LRAR_OK;
}

// Key mode of the block entry points.  Full-rank block sources are block
// AttnRes; by Sec. 3.4 sliced keys with r = d are exactly that, so they run
// as sliced keys over the whole row.
int block_keys(int *mode, int64_t d, int64_t r)
{
    if (*mode == LRAR_MODE_FULL) {
        if (r != d)
            return fail(LRAR_EINVAL, "full-rank keys need r == d");
        *mode = LRAR_MODE_SLICED;
        return LRAR_OK;
    }
    if (*mode != LRAR_MODE_PROJECTED && *mode != LRAR_MODE_SLICED)
        return fail(LRAR_EINVAL, "block routing takes projected, sliced or full-rank keys");
    return LRAR_OK;
}

}  // namespace

extern "C" {

int lr_attnres_route_fwd(const void *V, const void *K, const float *q, void *H, int64_t S,
                         int64_t N, int64_t d, int64_t r, int mode, int dtype, float eps,
                         void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(H, "H", 16, data)) ||
        (rc = check_ptr(K, "K", 16, data && mode == LRAR_MODE_PROJECTED)))
        return rc;
    if (mode != LRAR_MODE_PROJECTED && K)
        return fail(LRAR_EINVAL, "K must be NULL unless keys are projected");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    const Span outs[] = {span("H", H, he * es)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("q", q, r * 4)};
    if ((rc = check_aliasing(outs, 1, ins, 3)))
        return rc;
    lrar::Problem p{V, K, q, S, N, d, r, mode, dtype, eps, dtype};
    std::string why;
    if ((rc = lrar::check_supported(p, false, &why)))
        return fail(rc, why);
    if ((rc = lrar::launch_fwd(p, H, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

size_t lr_attnres_route_bwd_workspace_bytes(int64_t S, int64_t N, int64_t d, int64_t r,
                                            int mode, int dtype)
{
    int64_t ve, ke, he;
    const std::string saved = g_last_error;
    const int rc = check_shape(S, N, d, r, mode, dtype, 0.0f, &ve, &ke, &he);
    g_last_error = saved;
    if (rc)
        return 0;
    lrar::Problem p{nullptr, nullptr, nullptr, S, N, d, r, mode, dtype, 0.0f, dtype};
    return lrar::bwd_workspace_bytes(p);
}

}  // extern "C"

namespace {

// noalloc: the dq partials go to the library's own device array (workspace
// must then be NULL with size 0).
int route_bwd(const void *V, const void *K, const float *q, const void *dH, void *dV, void *dK,
              float *dq, void *workspace, size_t workspace_bytes, int64_t S, int64_t N, int64_t d,
              int64_t r, int mode, int dtype, float eps, bool accumulate, void *stream,
              bool noalloc = false)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(dH, "dH", 16, data)) || (rc = check_ptr(dV, "dV", 16, data)) ||
        (rc = check_ptr(dq, "dq", 4, true)) || (rc = check_ptr(K, "K", 16, data && proj)) ||
        (rc = check_ptr(dK, "dK", 16, data && proj)) ||
        (rc = check_ptr(workspace, "workspace", 16, false)))
        return rc;
    if (!proj && (K || dK))
        return fail(LRAR_EINVAL, "K and dK must be NULL unless keys are projected");
    lrar::Problem p{V, K, q, S, N, d, r, mode, dtype, eps, dtype};
    std::string why;
    if ((rc = lrar::check_supported(p, true, &why)))
        return fail(rc, why);
    const size_t need = noalloc ? 0 : lrar::bwd_workspace_bytes(p);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    const Span outs[] = {span("dV", dV, ve * es), span("dK", dK, ke * es),
                         span("dq", dq, r * 4), span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("q", q, r * 4),
                        span("dH", dH, he * es)};
    if ((rc = check_aliasing(outs, 4, ins, 4)))
        return rc;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (noalloc)
        rc = lrar::launch_bwd_noalloc(p, dH, dV, dK, dq, st, &why);
    else
        rc = lrar::launch_bwd(p, dH, dV, dK, dq, workspace, accumulate, st, &why);
    if (rc)
        return fail(rc, why);
    return LRAR_OK;
}

}  // namespace

extern "C" {

int lr_attnres_route_bwd(const void *V, const void *K, const float *q, const void *dH, void *dV,
                         void *dK, float *dq, void *workspace, size_t workspace_bytes,
                         int64_t S, int64_t N, int64_t d, int64_t r, int mode, int dtype,
                         float eps, void *stream)
{
    return route_bwd(V, K, q, dH, dV, dK, dq, workspace, workspace_bytes, S, N, d, r, mode, dtype,
                     eps, false, stream);
}

int lr_attnres_route_bwd_noalloc(const void *V, const void *K, const float *q, const void *dH,
                                 void *dV, void *dK, float *dq, int64_t S, int64_t N, int64_t d,
                                 int64_t r, int mode, int dtype, float eps, void *stream)
{
    return route_bwd(V, K, q, dH, dV, dK, dq, nullptr, 0, S, N, d, r, mode, dtype, eps, false,
                     stream, true);
}

int lr_attnres_route_bwd_accumulate(const void *V, const void *K, const float *q, const void *dH,
                                    void *dV, void *dK, float *dq, void *workspace,
                                    size_t workspace_bytes, int64_t S, int64_t N, int64_t d,
                                    int64_t r, int mode, int dtype, float eps, void *stream)
{
    return route_bwd(V, K, q, dH, dV, dK, dq, workspace, workspace_bytes, S, N, d, r, mode, dtype,
                     eps, true, stream);
}

int lr_attnres_block_route_fwd(float *B, float *KB, const void *o_new, const void *k_new,
                               const float *q, void *H, int64_t n_src, int start, int64_t N,
                               int64_t d, int64_t r, int mode, int dtype, float eps,
                               void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    if (start != 0 && start != 1)
        return fail(LRAR_EINVAL, "start must be 0 or 1");
    int64_t ve, ke, he;
    int rc = check_shape(n_src, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(o_new, "o_new", 16, data)) ||
        (rc = check_ptr(q, "q", 4, true)) || (rc = check_ptr(H, "H", 16, data)) ||
        (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(k_new, "k_new", (size_t)(dtype == LRAR_DTYPE_BF16 ? 2 : 4),
                        data && proj)))
        return rc;
    if (!proj && (KB || k_new))
        return fail(LRAR_EINVAL, "KB and k_new must be NULL unless keys are projected");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t nr;
    if (!mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    // B and KB are read and rewritten: checked as outputs.
    const Span outs[] = {span("H", H, he * es), span("B", B, ve * 4), span("KB", KB, ke * 4)};
    const Span ins[] = {span("o_new", o_new, he * es), span("k_new", k_new, nr * es),
                        span("q", q, r * 4)};
    if ((rc = check_aliasing(outs, 3, ins, 3)))
        return rc;
    lrar::BlockProblem p{B, KB, o_new, k_new, q, H, n_src, N, d, r, start, mode, dtype, eps};
    std::string why;
    if ((rc = lrar::check_block_supported(p, &why)))
        return fail(rc, why);
    if ((rc = lrar::launch_block_fwd(p, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_route_bwd(float *B, float *KB, float *dB, float *dKB, const void *o_new,
                               const void *k_new, const float *q, const void *dH, void *dO,
                               void *dK, float *dq, void *workspace, size_t workspace_bytes,
                               int64_t n_src, int64_t N, int64_t d, int64_t r, int mode,
                               int dtype, float eps, void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    int64_t ve, ke, he;
    int rc = check_shape(n_src, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const size_t ek = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(dB, "dB", 16, data)) ||
        (rc = check_ptr(o_new, "o_new", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(dH, "dH", 16, data)) || (rc = check_ptr(dO, "dO", 16, data)) ||
        (rc = check_ptr(dq, "dq", 4, true)) || (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(dKB, "dKB", 16, data && proj)) ||
        (rc = check_ptr(k_new, "k_new", ek, data && proj)) ||
        (rc = check_ptr(dK, "dK", ek, data && proj)) ||
        (rc = check_ptr(workspace, "workspace", 16, false)))
        return rc;
    if (!proj && (KB || dKB || k_new || dK))
        return fail(LRAR_EINVAL, "KB, dKB, k_new and dK must be NULL unless keys are projected");
    const lrar::BlockProblem bp{B, KB, o_new, k_new, q, nullptr, n_src, N, d, r, 0, mode,
                                dtype, eps};
    std::string why;
    if ((rc = lrar::check_block_supported(bp, &why)))
        return fail(rc, why);
    // The routing backward runs over the fp32 slots with the model-dtype dH.
    lrar::Problem p{B, KB, q, n_src, N, d, r, mode, LRAR_DTYPE_F32, eps, dtype};
    if ((rc = lrar::check_supported(p, true, &why)))
        return fail(rc, why);
    const size_t need = lrar::bwd_workspace_bytes(p);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t nr;
    if (!mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("B", B, ve * 4),         span("KB", KB, ke * 4),
                         span("dB", dB, ve * 4),       span("dKB", dKB, ke * 4),
                         span("dO", dO, he * es),      span("dK", dK, nr * es),
                         span("dq", dq, r * 4),        span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("o_new", o_new, he * es), span("k_new", k_new, nr * es),
                        span("q", q, r * 4), span("dH", dH, he * es)};
    if ((rc = check_aliasing(outs, 8, ins, 4)))
        return rc;
    const lrar::BlockRetire br{B, KB, dB, dKB, o_new, k_new, dO, dK, n_src - 1, N, d, r, mode,
                               dtype};
    if ((rc = lrar::launch_block_bwd(p, br, dH, dB, dKB, dq, workspace,
                                     static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_route_fwd_bf16c(float *B, float *KB, void *BC, void *KBC,
                                     const void *o_new, const void *k_new, const float *q,
                                     void *H, int64_t n_src, int start, int finish, int64_t N,
                                     int64_t d, int64_t r, int mode, float eps, void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    if (start != 0 && start != 1)
        return fail(LRAR_EINVAL, "start must be 0 or 1");
    if (finish != 0 && finish != 1)
        return fail(LRAR_EINVAL, "finish must be 0 or 1");
    const int dtype = LRAR_DTYPE_BF16;
    int64_t ve, ke, he;
    int rc = check_shape(n_src, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    // The copies are read for the completed slots (n_src > 1) and written
    // for slot n_src - 1 when it finishes.
    const bool copies = data && (n_src > 1 || finish);
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(o_new, "o_new", 16, data)) ||
        (rc = check_ptr(q, "q", 4, true)) || (rc = check_ptr(H, "H", 16, data)) ||
        (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(k_new, "k_new", 2, data && proj)) ||
        (rc = check_ptr(BC, "BC", 16, copies)) || (rc = check_ptr(KBC, "KBC", 16, copies && proj)))
        return rc;
    if (!proj && (KB || k_new || KBC))
        return fail(LRAR_EINVAL, "KB, k_new and KBC must be NULL unless keys are projected");
    int64_t nr;
    if (!mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    // B, KB, BC and KBC are read and rewritten: checked as outputs.
    const Span outs[] = {span("H", H, he * 2), span("B", B, ve * 4), span("KB", KB, ke * 4),
                         span("BC", BC, ve * 2), span("KBC", KBC, ke * 2)};
    const Span ins[] = {span("o_new", o_new, he * 2), span("k_new", k_new, nr * 2),
                        span("q", q, r * 4)};
    if ((rc = check_aliasing(outs, 5, ins, 3)))
        return rc;
    lrar::BlockProblem p{B, KB, o_new, k_new, q, H, n_src, N, d, r, start, mode, dtype, eps};
    p.completed_bf16 = 1;
    p.BC = BC;
    p.KBC = KBC;
    p.finish = finish;
    std::string why;
    if ((rc = lrar::check_block_supported(p, &why)))
        return fail(rc, why);
    if ((rc = lrar::launch_block_fwd(p, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_inter_fwd(const float *B, const float *KB, const float *Q, float *M,
                               float *L, float *ACC, int64_t n_prev, int64_t n_queries,
                               int64_t N, int64_t d, int64_t r, int mode, float eps,
                               void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    if (n_queries < 1)
        return fail(LRAR_EINVAL, "n_queries must be >= 1");
    int64_t ve, ke, he;
    int rc = check_shape(n_prev, N, d, r, mode, LRAR_DTYPE_F32, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(Q, "Q", 4, true)) ||
        (rc = check_ptr(M, "M", 4, data)) || (rc = check_ptr(L, "L", 4, data)) ||
        (rc = check_ptr(ACC, "ACC", 16, data)) || (rc = check_ptr(KB, "KB", 16, data && proj)))
        return rc;
    if (!proj && KB)
        return fail(LRAR_EINVAL, "KB must be NULL unless keys are projected");
    int64_t qn, qnd, qr;
    if (!mul_ok(n_queries, N, &qn) || !mul_ok(qn, d, &qnd) || !mul_ok(n_queries, r, &qr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("M", M, qn * 4), span("L", L, qn * 4), span("ACC", ACC, qnd * 4)};
    const Span ins[] = {span("B", B, ve * 4), span("KB", KB, ke * 4), span("Q", Q, qr * 4)};
    if ((rc = check_aliasing(outs, 3, ins, 3)))
        return rc;
    const lrar::BlockInterProblem p{B, KB, Q, M, L, ACC, n_prev, n_queries, N, d, r, mode, eps};
    std::string why;
    if ((rc = lrar::launch_block_inter(p, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_merge_fwd(float *B, float *KB, const void *o_new, const void *k_new,
                               const float *q, const float *M, const float *L, const float *ACC,
                               void *H, int64_t slot, int start, int64_t N, int64_t d, int64_t r,
                               int mode, int dtype, float eps, void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    if (start != 0 && start != 1)
        return fail(LRAR_EINVAL, "start must be 0 or 1");
    if (slot < 0)
        return fail(LRAR_EINVAL, "slot must be >= 0");
    int64_t ve, ke, he;
    int rc = check_shape(slot + 1, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const bool state = slot > 0;
    const size_t ek = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(o_new, "o_new", 16, data)) ||
        (rc = check_ptr(q, "q", 4, true)) || (rc = check_ptr(H, "H", 16, data)) ||
        (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(k_new, "k_new", ek, data && proj)) ||
        (rc = check_ptr(M, "M", 4, data && state)) || (rc = check_ptr(L, "L", 4, data && state)) ||
        (rc = check_ptr(ACC, "ACC", 16, data && state)))
        return rc;
    if (!proj && (KB || k_new))
        return fail(LRAR_EINVAL, "KB and k_new must be NULL unless keys are projected");
    if (!state && (M || L || ACC))
        return fail(LRAR_EINVAL, "slot 0 has no completed slots: M, L and ACC must be NULL");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t nr;
    if (!mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("H", H, he * es), span("B", B, ve * 4), span("KB", KB, ke * 4)};
    const Span ins[] = {span("o_new", o_new, he * es), span("k_new", k_new, nr * es),
                        span("q", q, r * 4), span("M", M, N * 4), span("L", L, N * 4),
                        span("ACC", ACC, he * 4)};
    if ((rc = check_aliasing(outs, 3, ins, 6)))
        return rc;
    lrar::BlockProblem p{B, KB, o_new, k_new, q, H, slot + 1, N, d, r, start, mode, dtype, eps};
    std::string why;
    if ((rc = lrar::launch_block_merge(p, state ? M : nullptr, state ? L : nullptr,
                                       state ? ACC : nullptr, static_cast<hipStream_t>(stream),
                                       &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_route_state_fwd(const void *V, const void *K, const float *q, float *M, float *L,
                               float *ACC, int64_t S, int64_t N, int64_t d, int64_t r,
                               int64_t chunk, int mode, int dtype, float eps, void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    if (chunk < 1)
        return fail(LRAR_EINVAL, "chunk must be >= 1");
    const int64_t P = (S + chunk - 1) / chunk;
    const bool data = N > 0;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(M, "M", 4, data)) || (rc = check_ptr(L, "L", 4, data)) ||
        (rc = check_ptr(ACC, "ACC", 16, data)) ||
        (rc = check_ptr(K, "K", 16, data && mode == LRAR_MODE_PROJECTED)))
        return rc;
    if (mode != LRAR_MODE_PROJECTED && K)
        return fail(LRAR_EINVAL, "K must be NULL unless keys are projected");
    int64_t pn, pnd;
    if (!mul_ok(P, N, &pn) || !mul_ok(pn, d, &pnd))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    const Span outs[] = {span("M", M, pn * 4), span("L", L, pn * 4), span("ACC", ACC, pnd * 4)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("q", q, r * 4)};
    if ((rc = check_aliasing(outs, 3, ins, 3)))
        return rc;
    // The plan (and the source limit) is that of one chunk.
    lrar::Problem p{V, K, q, S, N, d, r, mode, dtype, eps, dtype};
    std::string why;
    if ((rc = lrar::launch_state(p, chunk, M, L, ACC, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_route_merge_fwd(const float *M, const float *L, const float *ACC, void *H,
                               int64_t P, int64_t N, int64_t d, int dtype, void *stream)
{
    g_last_error.clear();
    if (P < 1)
        return fail(LRAR_EINVAL, "P must be >= 1");
    if (N < 0 || d < 1)
        return fail(LRAR_EINVAL, "need N >= 0 and d >= 1");
    if (dtype != LRAR_DTYPE_F32 && dtype != LRAR_DTYPE_BF16)
        return fail(LRAR_EINVAL, "dtype must be LRAR_DTYPE_F32 or LRAR_DTYPE_BF16");
    int rc;
    const bool data = N > 0;
    if ((rc = check_ptr(M, "M", 4, data)) || (rc = check_ptr(L, "L", 4, data)) ||
        (rc = check_ptr(ACC, "ACC", 16, data)) || (rc = check_ptr(H, "H", 16, data)))
        return rc;
    int64_t pn, pnd, nd;
    if (!mul_ok(P, N, &pn) || !mul_ok(pn, d, &pnd) || !mul_ok(N, d, &nd))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    const Span outs[] = {span("H", H, nd * es)};
    const Span ins[] = {span("M", M, pn * 4), span("L", L, pn * 4), span("ACC", ACC, pnd * 4)};
    if ((rc = check_aliasing(outs, 1, ins, 3)))
        return rc;
    std::string why;
    if ((rc = lrar::launch_merge(M, L, ACC, P, N, d, dtype, H, static_cast<hipStream_t>(stream),
                                 &why)))
        return fail(rc, why);
    return LRAR_OK;
}

const char *lr_attnres_last_error(void) { return g_last_error.c_str(); }

int lr_attnres_abi_version(void) { return LR_ATTNRES_ABI_VERSION; }

int lr_attnres_route_all_fwd(const void *V, const void *K, const float *Q, void *H, float *neff,
                             int64_t S, int64_t N, int64_t d, int64_t r, int64_t first,
                             int64_t T, int mode, int dtype, float eps, void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    if (first < 1 || T < 1 || first > S || T > S - first + 1)
        return fail(LRAR_EINVAL, "sites need first >= 1, T >= 1 and first + T - 1 <= S");
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(Q, "Q", 4, true)) ||
        (rc = check_ptr(H, "H", 16, data)) || (rc = check_ptr(K, "K", es, data && proj)) ||
        (rc = check_ptr(neff, "neff", 4, false)))
        return rc;
    if (!proj && K)
        return fail(LRAR_EINVAL, "K must be NULL unless keys are projected");
    int64_t tq, th, tn;
    if (!mul_ok(T, r, &tq) || !mul_ok(T, he, &th) || !mul_ok(th, es, &th) || !mul_ok(T, N, &tn))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("H", H, th), span("neff", neff, tn * 4)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("Q", Q, tq * 4)};
    if ((rc = check_aliasing(outs, 2, ins, 3)))
        return rc;
    lrar::AllProblem p{V, K, Q, H, neff, S, N, d, r, first, T, mode, dtype, eps};
    std::string why;
    if ((rc = lrar::check_all_supported(p, &why)))
        return fail(rc, why);
    if ((rc = lrar::launch_all_fwd(p, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

size_t lr_attnres_route_all_bwd_workspace_bytes(int64_t S, int64_t N, int64_t d, int64_t r,
                                                int64_t first, int64_t T, int mode, int dtype)
{
    int64_t ve, ke, he;
    const std::string saved = g_last_error;
    const int rc = check_shape(S, N, d, r, mode, dtype, 0.0f, &ve, &ke, &he);
    g_last_error = saved;
    if (rc || first < 1 || T < 1 || first > S || T > S - first + 1)
        return 0;
    lrar::AllProblem p{nullptr, nullptr, nullptr, nullptr, nullptr, S, N, d, r, first, T,
                       mode, dtype, 0.0f};
    return lrar::all_bwd_workspace_bytes(p);
}

int lr_attnres_route_all_bwd(const void *V, const void *K, const float *Q, const void *dH,
                             void *dV, void *dK, float *dQ, void *workspace,
                             size_t workspace_bytes, int64_t S, int64_t N, int64_t d, int64_t r,
                             int64_t first, int64_t T, int mode, int dtype, float eps,
                             int accumulate, void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    if (first < 1 || T < 1 || first > S || T > S - first + 1)
        return fail(LRAR_EINVAL, "sites need first >= 1, T >= 1 and first + T - 1 <= S");
    if (accumulate != 0 && accumulate != 1)
        return fail(LRAR_EINVAL, "accumulate must be 0 or 1");
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(Q, "Q", 4, true)) ||
        (rc = check_ptr(dH, "dH", 16, data)) || (rc = check_ptr(dV, "dV", 16, data)) ||
        (rc = check_ptr(dQ, "dQ", 4, true)) || (rc = check_ptr(K, "K", es, data && proj)) ||
        (rc = check_ptr(dK, "dK", es, data && proj)) ||
        (rc = check_ptr(workspace, "workspace", 4, false)))
        return rc;
    if (!proj && (K || dK))
        return fail(LRAR_EINVAL, "K and dK must be NULL unless keys are projected");
    int64_t tq, th;
    if (!mul_ok(T, r, &tq) || !mul_ok(T, he, &th) || !mul_ok(th, es, &th))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    lrar::AllProblem p{V, K, Q, nullptr, nullptr, S, N, d, r, first, T, mode, dtype, eps};
    std::string why;
    if ((rc = lrar::check_all_bwd_supported(p, &why)))
        return fail(rc, why);
    const size_t need = lrar::all_bwd_workspace_bytes(p);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const Span outs[] = {span("dV", dV, ve * es), span("dK", dK, ke * es),
                         span("dQ", dQ, tq * 4), span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("Q", Q, tq * 4),
                        span("dH", dH, th)};
    if ((rc = check_aliasing(outs, 4, ins, 4)))
        return rc;
    if ((rc = lrar::launch_all_bwd(p, dH, dV, dK, dQ, workspace, accumulate == 1,
                                   static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_key_proj_fwd(const void *A, const void *W, void *O, void *K, int64_t N,
                            int64_t m, int64_t d, int64_t r, int dtype, void *stream)
{
    g_last_error.clear();
    if (dtype != LRAR_DTYPE_F32 && dtype != LRAR_DTYPE_BF16)
        return fail(LRAR_EINVAL, "unknown storage type " + std::to_string(dtype));
    if (N < 0 || m < 1 || d < 0 || r < 0 || d + r < 1)
        return fail(LRAR_EINVAL, "sizes must satisfy N >= 0, m >= 1, d >= 0, r >= 0, d + r >= 1");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t ae, we, oe, ke;
    if (!mul_ok(N, m, &ae) || !mul_ok(d + r, m, &we) || !mul_ok(N, d, &oe) || !mul_ok(N, r, &ke) ||
        !mul_ok(ae, es, &ae) || !mul_ok(we, es, &we) || !mul_ok(oe, es, &oe) ||
        !mul_ok(ke, es, &ke))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const bool data = N > 0;
    int rc;
    if ((rc = check_ptr(A, "A", 16, data)) || (rc = check_ptr(W, "W", 16, data)) ||
        (rc = check_ptr(O, "O", es, data && d > 0)) || (rc = check_ptr(K, "K", es, data && r > 0)))
        return rc;
    if (d == 0 && O)
        return fail(LRAR_EINVAL, "O must be NULL when d = 0");
    if (r == 0 && K)
        return fail(LRAR_EINVAL, "K must be NULL when r = 0");
    const Span outs[] = {span("O", O, oe), span("K", K, ke)};
    const Span ins[] = {span("A", A, ae), span("W", W, we)};
    if ((rc = check_aliasing(outs, 2, ins, 2)))
        return rc;
    lrar::KeyProjProblem p{A, W, O, K, N, m, d, r, dtype};
    std::string why;
    if ((rc = lrar::check_key_proj_supported(p, &why)))
        return fail(rc, why);
    if ((rc = lrar::launch_key_proj(p, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

size_t lr_attnres_key_proj_bwd_workspace_bytes(int64_t N, int64_t m, int64_t d, int64_t r,
                                               int dtype)
{
    if (dtype != LRAR_DTYPE_BF16 || N < 0 || m < 1 || d < 0 || r < 0 || d + r < 1 ||
        N > ((int64_t)1 << 30) || m > (1 << 20) || d + r > (1 << 20))
        return 0;
    return lrar::key_proj_bwd_workspace_bytes(N, m, d, r);
}

int lr_attnres_key_proj_bwd(const void *A, const void *W, const void *dO, const void *dK,
                            void *dA, float *dW, void *workspace, size_t workspace_bytes,
                            int64_t N, int64_t m, int64_t d, int64_t r, int dtype, void *stream)
{
    g_last_error.clear();
    if (dtype != LRAR_DTYPE_F32 && dtype != LRAR_DTYPE_BF16)
        return fail(LRAR_EINVAL, "unknown storage type " + std::to_string(dtype));
    if (N < 0 || m < 1 || d < 0 || r < 0 || d + r < 1)
        return fail(LRAR_EINVAL, "sizes must satisfy N >= 0, m >= 1, d >= 0, r >= 0, d + r >= 1");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t ae, we, oe, ke, wf;
    if (!mul_ok(N, m, &ae) || !mul_ok(d + r, m, &we) || !mul_ok(N, d, &oe) || !mul_ok(N, r, &ke) ||
        !mul_ok(we, 4, &wf) || !mul_ok(ae, es, &ae) || !mul_ok(we, es, &we) ||
        !mul_ok(oe, es, &oe) || !mul_ok(ke, es, &ke))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const bool data = N > 0;
    int rc;
    if ((rc = check_ptr(A, "A", 16, data)) || (rc = check_ptr(W, "W", 16, data)) ||
        (rc = check_ptr(dO, "dO", 16, data && d > 0)) ||
        (rc = check_ptr(dK, "dK", 16, data && r > 0)) || (rc = check_ptr(dA, "dA", 16, data)) ||
        (rc = check_ptr(dW, "dW", 16, true)) || (rc = check_ptr(workspace, "workspace", 16, false)))
        return rc;
    if (d == 0 && dO)
        return fail(LRAR_EINVAL, "dO must be NULL when d = 0");
    if (r == 0 && dK)
        return fail(LRAR_EINVAL, "dK must be NULL when r = 0");
    lrar::KeyProjProblem p{A, W, nullptr, nullptr, N, m, d, r, dtype};
    std::string why;
    if ((rc = lrar::check_key_proj_bwd_supported(p, &why)))
        return fail(rc, why);
    const size_t need = lrar::key_proj_bwd_workspace_bytes(N, m, d, r);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const Span outs[] = {span("dA", dA, ae), span("dW", dW, wf),
                         span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("A", A, ae), span("W", W, we), span("dO", dO, oe),
                        span("dK", dK, ke)};
    if ((rc = check_aliasing(outs, 3, ins, 4)))
        return rc;
    if ((rc = lrar::launch_key_proj_bwd(p, dO, dK, dA, dW, workspace,
                                        static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_route_neff(const void *V, const void *K, const float *q, float *neff, int64_t S,
                          int64_t N, int64_t d, int64_t r, int mode, int dtype, float eps,
                          void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(V, "V", 16, data && !proj)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(neff, "neff", 4, data)) || (rc = check_ptr(K, "K", 16, data && proj)))
        return rc;
    if (!proj && K)
        return fail(LRAR_EINVAL, "K must be NULL unless keys are projected");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    const Span outs[] = {span("neff", neff, N * 4)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("q", q, r * 4)};
    if ((rc = check_aliasing(outs, 1, ins, 3)))
        return rc;
    // Full rank: the key is the whole value (Sec. 3.4: sliced keys with r = d).
    lrar::Problem p{V, K, q, S, N, d, r, mode == LRAR_MODE_FULL ? LRAR_MODE_SLICED : mode, dtype,
                    eps, dtype};
    std::string why;
    if ((rc = lrar::launch_neff(p, neff, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_route_bwd_deferred(float *B, float *KB, float *dP, float *dKP, float *coef,
                                        const void *o_new, const void *k_new, const float *q,
                                        const void *dH, void *dO, void *dK, float *dq,
                                        void *workspace, size_t workspace_bytes, int64_t n_src,
                                        int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                        float eps, void *stream)
{
    g_last_error.clear();
    if (int krc = block_keys(&mode, d, r))
        return krc;
    int64_t ve, ke, he;
    int rc = check_shape(n_src, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const size_t ek = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(dP, "dP", 16, data)) ||
        (rc = check_ptr(coef, "coef", 4, data && n_src > 1)) ||
        (rc = check_ptr(o_new, "o_new", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(dH, "dH", 16, data)) || (rc = check_ptr(dO, "dO", 16, data)) ||
        (rc = check_ptr(dq, "dq", 4, true)) || (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(dKP, "dKP", 16, data && proj)) ||
        (rc = check_ptr(k_new, "k_new", ek, data && proj)) ||
        (rc = check_ptr(dK, "dK", ek, data && proj)) ||
        (rc = check_ptr(workspace, "workspace", 16, false)))
        return rc;
    if (!proj && (KB || dKP || k_new || dK))
        return fail(LRAR_EINVAL, "KB, dKP, k_new and dK must be NULL unless keys are projected");
    const lrar::BlockProblem bp{B, KB, o_new, k_new, q, nullptr, n_src, N, d, r, 0, mode,
                                dtype, eps};
    std::string why;
    if ((rc = lrar::check_block_supported(bp, &why)))
        return fail(rc, why);
    lrar::Problem p{B, KB, q, n_src, N, d, r, mode, LRAR_DTYPE_F32, eps, dtype};
    if ((rc = lrar::check_supported(p, true, &why)))
        return fail(rc, why);
    const size_t need = lrar::bwd_workspace_bytes(p);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t nr, nc;
    if (!mul_ok(N, r, &nr) || !mul_ok(n_src - 1, 3 * N, &nc))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("B", B, ve * 4),    span("KB", KB, ke * 4),
                         span("dP", dP, he * 4),  span("dKP", dKP, nr * 4),
                         span("coef", coef, nc * 4), span("dO", dO, he * es),
                         span("dK", dK, nr * es), span("dq", dq, r * 4),
                         span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("o_new", o_new, he * es), span("k_new", k_new, nr * es),
                        span("q", q, r * 4), span("dH", dH, he * es)};
    if ((rc = check_aliasing(outs, 9, ins, 4)))
        return rc;
    lrar::BlockRetire br{B, KB, dP, dKP, o_new, k_new, dO, dK, n_src - 1, N, d, r, mode, dtype};
    br.grad_rows = true;
    if ((rc = lrar::launch_block_bwd_deferred(p, br, dH, dP, dKP, coef, dq, workspace,
                                              static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_route_bwd_deferred(const void *V, const void *K, const float *q, const void *dH,
                                  float *coef, float *dq, void *workspace, size_t workspace_bytes,
                                  int64_t S, int64_t N, int64_t d, int64_t r, int mode, int dtype,
                                  float eps, void *stream)
{
    g_last_error.clear();
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(q, "q", 4, true)) ||
        (rc = check_ptr(dH, "dH", 16, data)) || (rc = check_ptr(coef, "coef", 4, data)) ||
        (rc = check_ptr(dq, "dq", 4, true)) || (rc = check_ptr(K, "K", 16, data && proj)) ||
        (rc = check_ptr(workspace, "workspace", 16, false)))
        return rc;
    if (!proj && K)
        return fail(LRAR_EINVAL, "K must be NULL unless keys are projected");
    if (mode == LRAR_MODE_FULL)
        return fail(LRAR_EUNSUPPORTED, "the deferred backward takes projected or sliced keys");
    lrar::Problem p{V, K, q, S, N, d, r, mode, dtype, eps, dtype};
    std::string why;
    if ((rc = lrar::check_supported(p, true, &why)))
        return fail(rc, why);
    const size_t need = lrar::bwd_workspace_bytes(p);
    if (need > 0 && (!workspace || workspace_bytes < need))
        return fail(LRAR_EINVAL, "workspace too small: need " + std::to_string(need) + " bytes");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t nc;
    if (!mul_ok(S, 3 * N, &nc))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    const Span outs[] = {span("coef", coef, nc * 4), span("dq", dq, r * 4),
                         span("workspace", workspace, (int64_t)need)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("q", q, r * 4),
                        span("dH", dH, he * es)};
    if ((rc = check_aliasing(outs, 3, ins, 4)))
        return rc;
    if ((rc = lrar::launch_bwd_deferred_all(p, dH, coef, dq, workspace,
                                            static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_route_gather_bwd(const void *V, const void *K, int64_t source, const void *dHs,
                                const float *Q, const float *coef, int64_t coef_site_stride,
                                int64_t n_sites, void *dV, void *dK, int64_t S, int64_t N,
                                int64_t d, int64_t r, int mode, int dtype, float eps,
                                void *stream)
{
    g_last_error.clear();
    if (source < 0 || n_sites < 0)
        return fail(LRAR_EINVAL, "source and n_sites must be >= 0");
    int64_t ve, ke, he;
    int rc = check_shape(S, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    if (source >= S)
        return fail(LRAR_EINVAL, "source must be < S");
    if (mode == LRAR_MODE_FULL)
        return fail(LRAR_EUNSUPPORTED, "the source gather takes projected or sliced keys");
    if (n_sites > 0 && coef_site_stride < 3 * N)
        return fail(LRAR_EINVAL, "coef_site_stride must be at least 3 N");
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    if ((rc = check_ptr(V, "V", 16, data)) || (rc = check_ptr(dV, "dV", 16, data)) ||
        (rc = check_ptr(dHs, "dHs", 16, data && n_sites > 0)) ||
        (rc = check_ptr(Q, "Q", 4, n_sites > 0)) ||
        (rc = check_ptr(coef, "coef", 4, data && n_sites > 0)) ||
        (rc = check_ptr(K, "K", es, data && proj)) || (rc = check_ptr(dK, "dK", es, data && proj)))
        return rc;
    if (!proj && (K || dK))
        return fail(LRAR_EINVAL, "K and dK must be NULL unless keys are projected");
    int64_t hs, qn, cn, nr;
    if (!mul_ok(n_sites, he, &hs) || !mul_ok(hs, es, &hs) || !mul_ok(n_sites, r, &qn) ||
        !mul_ok(n_sites > 0 ? n_sites - 1 : 0, coef_site_stride, &cn) || !mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    cn = n_sites > 0 ? cn + 3 * N : 0;
    const Span outs[] = {span("dV", dV, he * es), span("dK", dK, nr * es)};
    const Span ins[] = {span("V", V, ve * es), span("K", K, ke * es), span("dHs", dHs, hs),
                        span("Q", Q, qn * 4), span("coef", coef, cn * 4)};
    if ((rc = check_aliasing(outs, 2, ins, 5)))
        return rc;
    lrar::BlockGather g{static_cast<const char *>(V) + source * he * es,
                        proj ? static_cast<const char *>(K) + source * nr * es : nullptr,
                        dHs, Q, coef, coef_site_stride, n_sites, dV, dK, N, d, r, mode, dtype, eps};
    g.kdtype = dtype;
    std::string why;
    if ((rc = lrar::launch_block_gather(g, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

int lr_attnres_block_gather_bwd(const float *B, const float *KB, int64_t slot, const void *dHs,
                                const float *Q, const float *coef, int64_t coef_site_stride,
                                int64_t n_sites, float *dP, float *dKP, int64_t N, int64_t d,
                                int64_t r, int mode, int dtype, float eps, void *stream)
{
    g_last_error.clear();
    if (slot < 0 || n_sites < 0)
        return fail(LRAR_EINVAL, "slot and n_sites must be >= 0");
    if (int krc = block_keys(&mode, d, r))
        return krc;
    int64_t ve, ke, he;
    int rc = check_shape(slot + 1, N, d, r, mode, dtype, eps, &ve, &ke, &he);
    if (rc)
        return rc;
    if (n_sites > 0 && coef_site_stride < 3 * N)
        return fail(LRAR_EINVAL, "coef_site_stride must be at least 3 N");
    const bool data = N > 0;
    const bool proj = mode == LRAR_MODE_PROJECTED;
    if ((rc = check_ptr(B, "B", 16, data)) || (rc = check_ptr(dP, "dP", 16, data)) ||
        (rc = check_ptr(dHs, "dHs", 16, data && n_sites > 0)) ||
        (rc = check_ptr(Q, "Q", 4, n_sites > 0)) ||
        (rc = check_ptr(coef, "coef", 4, data && n_sites > 0)) ||
        (rc = check_ptr(KB, "KB", 16, data && proj)) ||
        (rc = check_ptr(dKP, "dKP", 16, data && proj)))
        return rc;
    if (!proj && (KB || dKP))
        return fail(LRAR_EINVAL, "KB and dKP must be NULL unless keys are projected");
    const int64_t es = dtype == LRAR_DTYPE_BF16 ? 2 : 4;
    int64_t hs, qn, cn, nr;
    if (!mul_ok(n_sites, he, &hs) || !mul_ok(hs, es, &hs) || !mul_ok(n_sites, r, &qn) ||
        !mul_ok(n_sites > 0 ? n_sites - 1 : 0, coef_site_stride, &cn) || !mul_ok(N, r, &nr))
        return fail(LRAR_EINVAL, "tensor size overflows int64");
    cn = n_sites > 0 ? cn + 3 * N : 0;
    const Span outs[] = {span("dP", dP, he * 4), span("dKP", dKP, nr * 4)};
    const Span ins[] = {span("B", B, ve * 4), span("KB", KB, ke * 4), span("dHs", dHs, hs),
                        span("Q", Q, qn * 4), span("coef", coef, cn * 4)};
    if ((rc = check_aliasing(outs, 2, ins, 5)))
        return rc;
    const lrar::BlockGather g{B + slot * N * d, proj ? KB + slot * N * r : nullptr, dHs, Q, coef,
                              coef_site_stride, n_sites, dP, dKP, N, d, r, mode, dtype, eps};
    std::string why;
    if ((rc = lrar::launch_block_gather(g, static_cast<hipStream_t>(stream), &why)))
        return fail(rc, why);
    return LRAR_OK;
}

}  // extern "C"
