// Forward kernels of the LR-AttnRes depth routing (Sec. 3.2, Eqs.
// lr_key_norm, lr_attnres_weight, lr_attnres_output) and their launcher.
#include "route_common.h"

namespace lrar {

// ---------------------------------------------------------------------------
// Forward kernels
// ---------------------------------------------------------------------------

// Projected / sliced keys.  Grid: x = token groups of kWaves, y = column
// blocks of NCH*64*VEC (more than one only for very wide rows; each column
// block recomputes the cheap r-dimensional scores).
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_lr(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
             T *__restrict__ H, int S, int N, int d, int r, int krow, int koff, float eps,
             int s_pad)
{
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; this kernel has no workgroup barrier
    float *alpha = lds + wave * s_pad;
    lr_scores<T, VEC>(keys, q, S, N, r, krow, koff, eps, n, lane, alpha, nullptr);
    depth_softmax(alpha, alpha, S, lane);

    const int col = blockIdx.y * (NCH * kWaveSize * VEC) + lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;
    float acc[NCH][VEC];
    mix_rows<T, VEC, NCH, FULLCOLS>(V + (size_t)n * d + col, (size_t)N * d, S, alpha, ok, acc);
    store_row<T, VEC, NCH, FULLCOLS>(H + (size_t)n * d + col, ok, acc);
}

// Full-rank AttnRes in one pass over the rows: an online softmax over depth.
// Per batch of 4 sources the rows stay in registers while one batched wave
// reduction forms their sum(o^2) and q.o; the running maximum m, the
// normaliser l and the accumulator are rescaled only when m grows.  Reads
// every row once, like the low-rank kernels.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_full_1p(const T *__restrict__ V, const float *__restrict__ q, T *__restrict__ H,
                  int S, int N, int d, float eps)
{
    typedef typename Raw<T, VEC>::type raw_t;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; no workgroup barrier below

    const int col = lane * VEC;
    bool ok[NCH];
    float qv[NCH][VEC], acc[NCH][VEC];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        ok[c] = col + c * kWaveSize * VEC < d;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            qv[c][e] = (FULLCOLS || ok[c]) ? q[col + c * kWaveSize * VEC + e] : 0.0f;
            acc[c][e] = 0.0f;
        }
    }
    const size_t plane = (size_t)N * d;
    const T *vbase = V + (size_t)n * d + col;
    float m = -INFINITY, l = 0.0f;
    for (int i0 = 0; i0 < S; i0 += 4) {
        raw_t raw[4][NCH];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i0 + u < S)
#pragma unroll
                for (int c = 0; c < NCH; ++c)
                    if (FULLCOLS || ok[c])
                        raw[u][c] = load_stream<T, VEC, kNtLoad>(
                            vbase + (size_t)(i0 + u) * plane + c * kWaveSize * VEC);
        float part[8];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float a = 0.0f, b = 0.0f;
            if (i0 + u < S) {
#pragma unroll
                for (int c = 0; c < NCH; ++c) {
                    if (FULLCOLS || ok[c]) {
                        float x[VEC];
                        widen(raw[u][c], x);
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            a = fmaf(x[e], x[e], a);
                            b = fmaf(qv[c][e], x[e], b);
                        }
                    }
                }
            }
            part[u] = a;
            part[4 + u] = b;
        }
        const float tot = multi_sum<8>(part, lane);
        float sc[4];
        float mb = -INFINITY;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float ssq = lane_value<8>(tot, u);
            const float dot = lane_value<8>(tot, 4 + u);
            sc[u] = i0 + u < S ? dot / sqrtf(ssq / (float)d + eps) : -INFINITY;
            mb = fmaxf(mb, sc[u]);
        }
        if (mb > m) {  // wave-uniform
            const float scale = expf(m - mb);
            l *= scale;
#pragma unroll
            for (int c = 0; c < NCH; ++c)
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[c][e] *= scale;
            m = mb;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (i0 + u < S) {
                const float w = expf(sc[u] - m);
                l += w;
#pragma unroll
                for (int c = 0; c < NCH; ++c) {
                    if (FULLCOLS || ok[c]) {
                        float x[VEC];
                        widen(raw[u][c], x);
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            acc[c][e] = fmaf(w, x[e], acc[c][e]);
                    }
                }
            }
        }
    }
    const float inv = 1.0f / l;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] *= inv;
    store_row<T, VEC, NCH, FULLCOLS>(H + (size_t)n * d + col, ok, acc);
}

namespace {

template <typename T, int VEC>
hipError_t launch_fwd_t(const Problem &p, const Plan &pl, void *H, hipStream_t st)
{
    const T *V = static_cast<const T *>(p.V);
    const bool full = p.mode == LRAR_MODE_FULL;
    const T *keys = p.mode == LRAR_MODE_PROJECTED ? static_cast<const T *>(p.K) : V;
    const int krow = p.mode == LRAR_MODE_PROJECTED ? (int)p.r : (int)p.d;
    const int koff = p.mode == LRAR_MODE_SLICED ? (int)(p.d - p.r) : 0;
    return dispatch_chunks<VEC>(pl, [&](auto nch, auto fc) -> hipError_t {
        constexpr int NCH = decltype(nch)::value;
        constexpr bool FC = decltype(fc)::value;
        if (full) {
            hipLaunchKernelGGL((route_fwd_full_1p<T, VEC, NCH, FC>), dim3(pl.nblocks),
                               dim3(kBlock), 0, st, V, p.q, static_cast<T *>(H), (int)p.S,
                               (int)p.N, (int)p.d, p.eps);
        } else {
            hipLaunchKernelGGL((route_fwd_lr<T, VEC, NCH, FC>), dim3(pl.nblocks, pl.ysplit),
                               dim3(kBlock), pl.lds, st, V, keys, p.q, static_cast<T *>(H),
                               (int)p.S, (int)p.N, (int)p.d, (int)p.r, krow, koff, p.eps,
                               pl.s_pad);
        }
        return hipGetLastError();
    });
}

}  // namespace

int launch_fwd(const Problem &p, void *H, hipStream_t st, std::string *err)
{
    Plan pl;
    if (!make_plan(p, false, &pl, err))
        return LRAR_EUNSUPPORTED;
    if (p.N == 0)
        return LRAR_OK;
    hipError_t e;
    if (p.dtype == LRAR_DTYPE_BF16)
        e = pl.vec > 1 ? launch_fwd_t<uint16_t, 8>(p, pl, H, st)
                       : launch_fwd_t<uint16_t, 1>(p, pl, H, st);
    else
        e = pl.vec > 1 ? launch_fwd_t<float, 4>(p, pl, H, st) : launch_fwd_t<float, 1>(p, pl, H, st);
    return hip_status(e, "route_fwd launch", err);
}

}  // namespace lrar
