// Block-source routing forward: Block AttnRes summaries (Sec. 3.1, Eqs.
// block_attnres_sum and block_attnres_partial_sum) routed with the low-rank
// keys of Sec. 3.2.
//
// The summaries live in fp32 slots [slot][N][d]: slot 0 holds the embedding,
// slot j >= 1 the sum of block j's outputs written so far (its partial sum
// while the block is in progress).  One call serves one residual site: it
// adds the newest sub-layer output o_new (model storage) into its block's
// slot j = n_src - 1, or starts that slot with it, keeps the updated row in
// registers, and routes over slots 0..j: the earlier slots stream from HBM,
// slot j comes from the registers.  A summary's key is the sum of its
// members' keys: for sliced keys the tail of the summed row, for projected
// keys a second fp32 slot stack [slot][N][r] updated the same way.
#include <algorithm>

#include "route_common.h"

namespace lrar {

template <typename TO, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_block(float *__restrict__ B, float *__restrict__ KB, const TO *__restrict__ o_new,
                const TO *__restrict__ k_new, const float *__restrict__ q, TO *__restrict__ H,
                int nsrc, int start, int N, int d, int r, int sliced, float eps, int s_pad)
{
    constexpr int VEC = 4;  // fp32 slot rows move in 16-byte vectors of 4
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; no workgroup barrier below
    float *s = lds + wave * s_pad;  // scores, then weights
    const int j = nsrc - 1;
    const size_t plane = (size_t)N * d;
    const int col = lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;

    // 1. The updated summary row of slot j (Eqs. block_attnres_sum /
    //    block_attnres_partial_sum: one more member added), kept in registers.
    float nw[NCH][VEC];
    float *brow = B + (size_t)j * plane + (size_t)n * d + col;
    const TO *orow = o_new + (size_t)n * d + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (FULLCOLS || ok[c]) {
            float x[VEC];
            widen(load_raw<TO, VEC>(orow + c * kWaveSize * VEC), x);
            if (!start) {
                float b[VEC];
                widen(load_raw<float, VEC>(brow + c * kWaveSize * VEC), b);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    x[e] += b[e];
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nw[c][e] = x[e];
            store_raw<float, VEC>(brow + c * kWaveSize * VEC, Narrow<float, VEC>::run(nw[c]));
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nw[c][e] = 0.0f;
        }
    }

    // 2. Score of slot j from its updated key (Eqs. lr_key_norm, lr_attnres_weight).
    float ss = 0.0f, dot = 0.0f;
    if (sliced) {
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const int cc = col + c * kWaveSize * VEC + e;
                if ((FULLCOLS || ok[c]) && cc >= d - r) {
                    ss = fmaf(nw[c][e], nw[c][e], ss);
                    dot = fmaf(q[cc - (d - r)], nw[c][e], dot);
                }
            }
    } else {
        float *krow = KB + ((size_t)j * N + n) * r;
        const TO *knew = k_new + (size_t)n * r;
        for (int jj = lane; jj < r; jj += kWaveSize) {
            const float k = (start ? 0.0f : krow[jj]) + load_elem(knew + jj);
            krow[jj] = k;
            ss = fmaf(k, k, ss);
            dot = fmaf(q[jj], k, dot);
        }
    }
    ss = wave_sum(ss);
    dot = wave_sum(dot);
    const float sj = dot / sqrtf(ss / (float)r + eps);

    // 3. Scores of the earlier slots, lane per slot, from their fp32 keys.
    lr_scores<float, VEC>(sliced ? B : KB, q, j, N, r, sliced ? d : r, sliced ? d - r : 0, eps,
                          n, lane, s, nullptr);
    if (lane == 0)
        s[j] = sj;
    wave_lds_sync();
    depth_softmax(s, s, nsrc, lane);

    // 4. h = sum_i alpha_i b_i: slots 0..j-1 from HBM, slot j from registers.
    float acc[NCH][VEC];
    mix_rows<float, VEC, NCH, FULLCOLS>(B + (size_t)n * d + col, plane, j, s, ok, acc);
    const float aj = s[j];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] = fmaf(aj, nw[c][e], acc[c][e]);
    TO *hrow = H + (size_t)n * d + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        if (FULLCOLS || ok[c])
            store_stream<TO, VEC, kNtStore>(hrow + c * kWaveSize * VEC,
                                            Narrow<TO, VEC>::run(acc[c]));
}

// Retire the member o_new from slot j and hand it its gradient (see
// BlockRetire): 4 consecutive row elements per thread, grid-stride.
template <typename TO>
__global__ void __launch_bounds__(256)
block_retire(float *__restrict__ Bj, const float *__restrict__ dBj, const TO *__restrict__ o_new,
             TO *__restrict__ dO, long long nvec)
{
    const long long stride = (long long)gridDim.x * 256;
    for (long long v = (long long)blockIdx.x * 256 + threadIdx.x; v < nvec; v += stride) {
        const long long e0 = v * 4;
        float b[4], o[4], g[4];
        widen(load_raw<float, 4>(Bj + e0), b);
        widen(load_raw<TO, 4>(o_new + e0), o);
        widen(load_raw<float, 4>(dBj + e0), g);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            b[e] -= o[e];
        store_raw<float, 4>(Bj + e0, Narrow<float, 4>::run(b));
        store_raw<TO, 4>(dO + e0, Narrow<TO, 4>::run(g));
    }
}

// The same for the projected key rows (any r): one element per thread.
template <typename TO>
__global__ void __launch_bounds__(256)
block_retire_keys(float *__restrict__ KBj, const float *__restrict__ dKBj,
                  const TO *__restrict__ k_new, TO *__restrict__ dK, long long n)
{
    const long long stride = (long long)gridDim.x * 256;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) {
        KBj[i] -= load_elem(k_new + i);
        store_elem(dK + i, dKBj[i]);
    }
}

template <typename TO>
hipError_t launch_retire_t(const BlockRetire &br, hipStream_t st)
{
    const size_t plane = (size_t)br.N * br.d;
    const long long nvec = (long long)(plane / 4);
    const int grid = (int)std::min<long long>((nvec + 255) / 256, 8192);
    hipLaunchKernelGGL(block_retire<TO>, dim3(grid), dim3(256), 0, st, br.B + br.j * plane,
                       br.dB + br.j * plane, static_cast<const TO *>(br.o_new),
                       static_cast<TO *>(br.dO), nvec);
    if (br.mode == LRAR_MODE_PROJECTED) {
        const size_t kplane = (size_t)br.N * br.r;
        const int kgrid = (int)std::min<long long>(((long long)kplane + 255) / 256, 8192);
        hipLaunchKernelGGL(block_retire_keys<TO>, dim3(kgrid), dim3(256), 0, st,
                           br.KB + br.j * kplane, br.dKB + br.j * kplane,
                           static_cast<const TO *>(br.k_new), static_cast<TO *>(br.dK),
                           (long long)kplane);
    }
    return hipGetLastError();
}

namespace {

template <typename TO>
hipError_t launch_block_t(const BlockProblem &p, int nch, bool fullcols, size_t lds, int nblocks,
                          hipStream_t st)
{
    const int s_pad = (int)((p.nsrc + 3) / 4 * 4);
    const int sliced = p.mode == LRAR_MODE_SLICED ? 1 : 0;
    auto go = [&](auto nchc, auto fc) {
        constexpr int NCH = decltype(nchc)::value;
        constexpr bool FC = decltype(fc)::value;
        hipLaunchKernelGGL((route_fwd_block<TO, NCH, FC>), dim3(nblocks), dim3(kBlock), lds, st,
                           p.B, p.KB, static_cast<const TO *>(p.o_new),
                           static_cast<const TO *>(p.k_new), p.q, static_cast<TO *>(p.H),
                           (int)p.nsrc, p.start, (int)p.N, (int)p.d, (int)p.r, sliced, p.eps,
                           s_pad);
        return hipGetLastError();
    };
    typedef std::true_type Y;
    typedef std::false_type F;
    switch (nch) {
    case 1: return fullcols ? go(std::integral_constant<int, 1>{}, Y{}) : go(std::integral_constant<int, 1>{}, F{});
    case 2: return fullcols ? go(std::integral_constant<int, 2>{}, Y{}) : go(std::integral_constant<int, 2>{}, F{});
    case 4: return fullcols ? go(std::integral_constant<int, 4>{}, Y{}) : go(std::integral_constant<int, 4>{}, F{});
    case 8: return fullcols ? go(std::integral_constant<int, 8>{}, Y{}) : go(std::integral_constant<int, 8>{}, F{});
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_block_retire(const BlockRetire &br, hipStream_t st)
{
    return br.dtype == LRAR_DTYPE_BF16 ? launch_retire_t<uint16_t>(br, st)
                                       : launch_retire_t<float>(br, st);
}

int check_block_supported(const BlockProblem &p, std::string *why)
{
    if (p.d % 4 != 0) {
        *why = "block routing needs d to be a multiple of 4";
        return LRAR_EUNSUPPORTED;
    }
    if (p.d > 2048) {
        *why = "block routing supports d <= 2048";
        return LRAR_EUNSUPPORTED;
    }
    if (p.nsrc > 1024) {
        *why = "block routing supports at most 1024 sources";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N > (1 << 30)) {
        *why = "N exceeds 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_block_fwd(const BlockProblem &p, hipStream_t st, std::string *err)
{
    int rc = check_block_supported(p, err);
    if (rc)
        return rc;
    if (p.N == 0)
        return LRAR_OK;
    const int need = (int)((p.d + 255) / 256);
    int nch = 1;
    while (nch < need)
        nch <<= 1;
    const bool fullcols = p.d % (256 * nch) == 0;
    const size_t lds = (size_t)kWaves * ((p.nsrc + 3) / 4 * 4) * sizeof(float);
    const int nblocks = (int)((p.N + kWaves - 1) / kWaves);
    const hipError_t e =
        p.dtype == LRAR_DTYPE_BF16
            ? launch_block_t<uint16_t>(p, nch, fullcols, lds, nblocks, st)
            : launch_block_t<float>(p, nch, fullcols, lds, nblocks, st);
    return hip_status(e, "block_route_fwd launch", err);
}

}  // namespace lrar
