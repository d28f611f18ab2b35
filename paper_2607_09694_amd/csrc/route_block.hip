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
//
// Completed summaries in bf16 (TC = bf16, a storage option): the earlier
// slots are read from bf16 copies BC [slot][N][d] (and KBC [slot][N][r])
// instead of the fp32 slots, which halves what a site reads of them; the
// partial slot stays fp32.  When `finish` is set, the call that adds a
// block's last member also writes that slot's copy: the updated fp32 row,
// rounded once to bf16.  With TC = float, BC and KBC are the fp32 slots
// themselves and nothing is written to them beyond the slot update.
#include <algorithm>
#include <type_traits>

#include "route_common.h"

namespace lrar {

template <typename TO, typename TC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_block(float *__restrict__ B, float *__restrict__ KB, TC *BC, TC *KBC,
                const TO *__restrict__ o_new, const TO *__restrict__ k_new,
                const float *__restrict__ q, TO *__restrict__ H, int nsrc, int start, int finish,
                int N, int d, int r, int sliced, float eps, int s_pad)
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

    // 1. Issue the loads of the new member and of slot j's row; they stay in
    //    flight while the earlier slots are scored.
    typedef typename Raw<TO, VEC>::type oraw_t;
    typedef typename Raw<float, VEC>::type braw_t;
    float *brow = B + (size_t)j * plane + (size_t)n * d + col;
    const TO *orow = o_new + (size_t)n * d + col;
    oraw_t oraw[NCH];
    braw_t braw[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (FULLCOLS || ok[c]) {
            oraw[c] = load_raw<TO, VEC>(orow + c * kWaveSize * VEC);
            if (!start)
                braw[c] = load_raw<float, VEC>(brow + c * kWaveSize * VEC);
        }
    }

    // 2. Scores of the earlier (completed) slots from their keys.
    lr_scores<TC, VEC>(sliced ? BC : KBC, q, j, N, r, sliced ? d : r, sliced ? d - r : 0, eps, n,
                       lane, s, nullptr);

    // 3. The updated summary row of slot j (Eqs. block_attnres_sum /
    //    block_attnres_partial_sum: one more member added), kept in registers,
    //    and its score (Eqs. lr_key_norm, lr_attnres_weight).
    float nw[NCH][VEC];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (FULLCOLS || ok[c]) {
            float x[VEC];
            widen(oraw[c], x);
            if (!start) {
                float b[VEC];
                widen(braw[c], b);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    x[e] += b[e];
            }
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nw[c][e] = x[e];
            store_raw<float, VEC>(brow + c * kWaveSize * VEC, Narrow<float, VEC>::run(nw[c]));
            if constexpr (!std::is_same<TC, float>::value)
                if (finish)
                    store_raw<TC, VEC>(BC + (size_t)j * plane + (size_t)n * d + col +
                                           c * kWaveSize * VEC,
                                       Narrow<TC, VEC>::run(nw[c]));
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nw[c][e] = 0.0f;
        }
    }
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
            const float kn = load_elem(knew + jj);
            const float k = start ? kn : krow[jj] + kn;  // from the first member, as the rows
            krow[jj] = k;
            if constexpr (!std::is_same<TC, float>::value)
                if (finish)
                    store_elem(KBC + ((size_t)j * N + n) * r + jj, k);
            ss = fmaf(k, k, ss);
            dot = fmaf(q[jj], k, dot);
        }
    }
    ss = wave_sum_t<true>(ss);
    dot = wave_sum_t<true>(dot);
    if (lane == 0)
        s[j] = dot / sqrtf(ss / (float)r + eps);
    wave_lds_sync();
    depth_softmax<true>(s, s, nsrc, lane);

    // 4. h = sum_i alpha_i b_i: slots 0..j-1 from HBM, slot j from registers.
    float acc[NCH][VEC];
    mix_rows<TC, VEC, NCH, FULLCOLS>(BC + (size_t)n * d + col, plane, j, s, ok, acc);
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

// ---------------------------------------------------------------------------
// Two-phase block inference (Sec. 3.5): the site queries do not depend on
// the input, so the c sites of one block can route over the completed slots
// together (phase 1); each site then adds the partial block it reads and
// merges it into that state with an online-softmax update (phase 2).
// ---------------------------------------------------------------------------

// Unnormalised softmax of one query over S scores in place:
// s_i <- exp(s_i - m), returns m = max_i s_i and *l = sum_i exp(s_i - m).
__device__ inline float partial_softmax(float *s, int S, int lane, float *l)
{
    float m = -INFINITY;
    for (int i = lane; i < S; i += kWaveSize)
        m = fmaxf(m, s[i]);
    m = wave_max_t<true>(m);
    float z = 0.0f;
    for (int i = lane; i < S; i += kWaveSize) {
        const float e = expf(s[i] - m);
        s[i] = e;
        z += e;
    }
    *l = wave_sum_t<true>(z);
    return m;
}

// Phase 1: for nq queries, the online-softmax state over the nprev completed
// slots: M[q][n] = max score, L[q][n] = sum exp(s - M), ACC[q][n][:] =
// sum exp(s - M) b_i.  Queries go in groups of QG; each slot row is read once
// per group.  Grid: x = token groups, y = column blocks of NCH*256 (each
// recomputes the cheap r-dimensional scores).
template <int NCH, int QG, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_block_inter(const float *__restrict__ B, const float *__restrict__ KB,
                  const float *__restrict__ Qs, float *__restrict__ M, float *__restrict__ L,
                  float *__restrict__ ACC, int nprev, int nq, int N, int d, int r, int sliced,
                  float eps, int s_pad)
{
    constexpr int VEC = 4;
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; no workgroup barrier below
    float *sc = lds + (size_t)wave * QG * s_pad;  // [QG][s_pad]
    const int col = blockIdx.y * (NCH * kWaveSize * VEC) + lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;
    const size_t plane = (size_t)N * d;
    const float *keys = sliced ? B : KB;
    const int krow = sliced ? d : r, koff = sliced ? d - r : 0;

    for (int q0 = 0; q0 < nq; q0 += QG) {
        const int qg = nq - q0 < QG ? nq - q0 : QG;
        float mq[QG], lq[QG];
#pragma unroll
        for (int u = 0; u < QG; ++u) {
            mq[u] = -INFINITY;
            lq[u] = 0.0f;
            if (u < qg) {
                lr_scores<float, VEC>(keys, Qs + (size_t)(q0 + u) * r, nprev, N, r, krow, koff,
                                      eps, n, lane, sc + u * s_pad, nullptr);
                mq[u] = partial_softmax(sc + u * s_pad, nprev, lane, &lq[u]);
            }
        }
        wave_lds_sync();
        float acc[QG][NCH][VEC];
#pragma unroll
        for (int u = 0; u < QG; ++u)
#pragma unroll
            for (int c = 0; c < NCH; ++c)
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[u][c][e] = 0.0f;
        const float *vbase = B + (size_t)n * d + col;
        for (int i = 0; i < nprev; ++i) {
            float x[NCH][VEC];
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULLCOLS || ok[c]) {
                    widen(load_stream<float, VEC, kNtLoad>(vbase + (size_t)i * plane +
                                                           c * kWaveSize * VEC), x[c]);
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        x[c][e] = 0.0f;
                }
            }
#pragma unroll
            for (int u = 0; u < QG; ++u) {
                if (u < qg) {
                    const float w = sc[u * s_pad + i];
#pragma unroll
                    for (int c = 0; c < NCH; ++c)
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            acc[u][c][e] = fmaf(w, x[c][e], acc[u][c][e]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < QG; ++u) {
            if (u < qg) {
                float *arow = ACC + (size_t)(q0 + u) * plane + (size_t)n * d + col;
#pragma unroll
                for (int c = 0; c < NCH; ++c)
                    if (FULLCOLS || ok[c])
                        store_raw<float, VEC>(arow + c * kWaveSize * VEC,
                                              Narrow<float, VEC>::run(acc[u][c]));
                if (blockIdx.y == 0 && lane == 0) {
                    M[(size_t)(q0 + u) * N + n] = mq[u];
                    L[(size_t)(q0 + u) * N + n] = lq[u];
                }
            }
        }
        wave_lds_sync();  // the next group reuses sc
    }
}

// Phase 2 at one site: slot j = `slot` (the partial block) gains o_new as in
// route_fwd_block; its score merges into the site's phase-1 state:
//   m' = max(M, s_j),  h = (e^{M-m'} ACC + e^{s_j-m'} b_j) / (e^{M-m'} L + e^{s_j-m'}).
// Without completed slots (has_state = 0) the state is empty and h = b_j.
template <typename TO, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_block_merge(float *__restrict__ B, float *__restrict__ KB, const TO *__restrict__ o_new,
                  const TO *__restrict__ k_new, const float *__restrict__ q,
                  const float *__restrict__ Ms, const float *__restrict__ Ls,
                  const float *__restrict__ ACC, TO *__restrict__ H, int slot, int start,
                  int has_state, int N, int d, int r, int sliced, float eps)
{
    constexpr int VEC = 4;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform
    const int j = slot;
    const size_t plane = (size_t)N * d;
    const int col = lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;

    float nw[NCH][VEC], st[NCH][VEC];
    float *brow = B + (size_t)j * plane + (size_t)n * d + col;
    const TO *orow = o_new + (size_t)n * d + col;
    const float *arow = has_state ? ACC + (size_t)n * d + col : nullptr;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (FULLCOLS || ok[c]) {
            float x[VEC];
            widen(load_raw<TO, VEC>(orow + c * kWaveSize * VEC), x);
            if (has_state)
                widen(load_stream<float, VEC, kNtLoad>(arow + c * kWaveSize * VEC), st[c]);
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
        }
        if (!has_state || !(FULLCOLS || ok[c])) {
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                st[c][e] = 0.0f;
        }
        if (!(FULLCOLS || ok[c])) {
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                nw[c][e] = 0.0f;
        }
    }

    // Score of the updated partial slot (as in route_fwd_block).
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
            const float kn = load_elem(knew + jj);
            const float k = start ? kn : krow[jj] + kn;  // from the first member, as the rows
            krow[jj] = k;
            ss = fmaf(k, k, ss);
            dot = fmaf(q[jj], k, dot);
        }
    }
    ss = wave_sum_t<true>(ss);
    dot = wave_sum_t<true>(dot);
    const float sj = dot / sqrtf(ss / (float)r + eps);

    const float m = has_state ? Ms[n] : -INFINITY;
    const float l = has_state ? Ls[n] : 0.0f;
    const float mm = fmaxf(m, sj);
    const float e1 = has_state ? expf(m - mm) : 0.0f;
    const float e2 = expf(sj - mm);
    const float inv = 1.0f / (e1 * l + e2);
    TO *hrow = H + (size_t)n * d + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (FULLCOLS || ok[c]) {
            float y[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                y[e] = fmaf(e1, st[c][e], e2 * nw[c][e]) * inv;
            store_stream<TO, VEC, kNtStore>(hrow + c * kWaveSize * VEC, Narrow<TO, VEC>::run(y));
        }
    }
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
                       br.dB + (br.grad_rows ? 0 : br.j * plane),
                       static_cast<const TO *>(br.o_new), static_cast<TO *>(br.dO), nvec);
    if (br.mode == LRAR_MODE_PROJECTED) {
        const size_t kplane = (size_t)br.N * br.r;
        const int kgrid = (int)std::min<long long>(((long long)kplane + 255) / 256, 8192);
        hipLaunchKernelGGL(block_retire_keys<TO>, dim3(kgrid), dim3(256), 0, st,
                           br.KB + br.j * kplane, br.dKB + (br.grad_rows ? 0 : br.j * kplane),
                           static_cast<const TO *>(br.k_new), static_cast<TO *>(br.dK),
                           (long long)kplane);
    }
    return hipGetLastError();
}

namespace {

template <typename TO, typename TC>
hipError_t launch_block_t(const BlockProblem &p, int nch, bool fullcols, size_t lds, int nblocks,
                          hipStream_t st)
{
    const int s_pad = (int)((p.nsrc + 3) / 4 * 4);
    const int sliced = p.mode == LRAR_MODE_SLICED ? 1 : 0;
    // fp32 completed slots are the slots themselves.
    TC *BC = std::is_same<TC, float>::value ? reinterpret_cast<TC *>(p.B) : static_cast<TC *>(p.BC);
    TC *KBC = std::is_same<TC, float>::value ? reinterpret_cast<TC *>(p.KB)
                                             : static_cast<TC *>(p.KBC);
    auto go = [&](auto nchc, auto fc) {
        constexpr int NCH = decltype(nchc)::value;
        constexpr bool FC = decltype(fc)::value;
        hipLaunchKernelGGL((route_fwd_block<TO, TC, NCH, FC>), dim3(nblocks), dim3(kBlock), lds,
                           st, p.B, p.KB, BC, KBC, static_cast<const TO *>(p.o_new),
                           static_cast<const TO *>(p.k_new), p.q, static_cast<TO *>(p.H),
                           (int)p.nsrc, p.start, p.finish, (int)p.N, (int)p.d, (int)p.r, sliced,
                           p.eps, s_pad);
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

int launch_block_inter(const BlockInterProblem &p, hipStream_t st, std::string *err)
{
    if (p.d % 4 != 0) {
        *err = "block routing needs d to be a multiple of 4";
        return LRAR_EUNSUPPORTED;
    }
    if (p.nprev > 1024 || p.nq > 64) {
        *err = "two-phase block routing supports at most 1024 completed slots and 64 queries";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N > (1 << 30)) {
        *err = "N exceeds 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N == 0)
        return LRAR_OK;
    const int need = (int)((p.d + 255) / 256);
    int nch = 1;
    while (nch < need && nch < 4)
        nch <<= 1;
    const int ysplit = (need + nch - 1) / nch;
    const bool fullcols = p.d % (256 * nch) == 0;
    const int s_pad = (int)((p.nprev + 3) / 4 * 4);
    const int nblocks = (int)((p.N + kWaves - 1) / kWaves);
    const int sliced = p.mode == LRAR_MODE_SLICED ? 1 : 0;
    auto go = [&](auto nchc, auto fc) {
        constexpr int NCH = decltype(nchc)::value;
        constexpr bool FC = decltype(fc)::value;
        constexpr int QG = NCH >= 4 ? 4 : 8;
        const size_t lds = (size_t)kWaves * QG * s_pad * sizeof(float);
        hipLaunchKernelGGL((route_block_inter<NCH, QG, FC>), dim3(nblocks, ysplit), dim3(kBlock),
                           lds, st, p.B, p.KB, p.Q, p.M, p.L, p.ACC, (int)p.nprev, (int)p.nq,
                           (int)p.N, (int)p.d, (int)p.r, sliced, p.eps, s_pad);
        return hipGetLastError();
    };
    typedef std::true_type Y;
    typedef std::false_type F;
    hipError_t e;
    switch (nch) {
    case 1: e = fullcols ? go(std::integral_constant<int, 1>{}, Y{}) : go(std::integral_constant<int, 1>{}, F{}); break;
    case 2: e = fullcols ? go(std::integral_constant<int, 2>{}, Y{}) : go(std::integral_constant<int, 2>{}, F{}); break;
    default: e = fullcols ? go(std::integral_constant<int, 4>{}, Y{}) : go(std::integral_constant<int, 4>{}, F{}); break;
    }
    return hip_status(e, "block_inter_fwd launch", err);
}

template <typename TO>
hipError_t launch_merge_t(const BlockProblem &p, const float *Ms, const float *Ls,
                          const float *ACC, int nch, bool fullcols, int nblocks, hipStream_t st)
{
    const int sliced = p.mode == LRAR_MODE_SLICED ? 1 : 0;
    const int has_state = Ms != nullptr;
    auto go = [&](auto nchc, auto fc) {
        constexpr int NCH = decltype(nchc)::value;
        constexpr bool FC = decltype(fc)::value;
        hipLaunchKernelGGL((route_block_merge<TO, NCH, FC>), dim3(nblocks), dim3(kBlock), 0, st,
                           p.B, p.KB, static_cast<const TO *>(p.o_new),
                           static_cast<const TO *>(p.k_new), p.q, Ms, Ls, ACC,
                           static_cast<TO *>(p.H), (int)(p.nsrc - 1), p.start, has_state,
                           (int)p.N, (int)p.d, (int)p.r, sliced, p.eps);
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

int launch_block_merge(const BlockProblem &p, const float *Ms, const float *Ls, const float *ACC,
                       hipStream_t st, std::string *err)
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
    const int nblocks = (int)((p.N + kWaves - 1) / kWaves);
    const hipError_t e =
        p.dtype == LRAR_DTYPE_BF16
            ? launch_merge_t<uint16_t>(p, Ms, Ls, ACC, nch, fullcols, nblocks, st)
            : launch_merge_t<float>(p, Ms, Ls, ACC, nch, fullcols, nblocks, st);
    return hip_status(e, "block_merge_fwd launch", err);
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

// ---------------------------------------------------------------------------
// Deferred reverse pass: the gradient of a completed slot j from the sites
// that read it as completed, formed once.  Each of those sites stored, per
// token, alpha_{t,j}, cq = ds/rho and ck = ds s / (rho r) (route_bwd_lr's
// deferred form), so that
//     dB_j = sum_t alpha_{t,j} dH_t      (every column)
//          + sum_t cq_t q_t - (sum_t ck_t) kbar_j   (the key columns),
// kbar_j = k_j / rho_j recomputed from the summary's key.  One wave per
// token streams the sites' dH rows like the forward's value stream.
// ---------------------------------------------------------------------------

struct GatherArgs {
    const void *Bj, *KBj;  // the source's rows [N][d] and key rows [N][r], storage TK
    const void *dHs;
    const float *Q, *coef;
    long long site_stride;
    void *dP, *dKP;        // its gradient rows, storage TK
    int n_sites, N, d, r, sliced, s_pad;
    float eps;
};

// TK: storage of the source rows read for the key and of the gradient rows
// written (fp32 for block summaries, the model dtype for the sources of a
// full-source pass); TH: storage of dH.
template <typename TK, typename TH, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock) block_gather(GatherArgs a)
{
    extern __shared__ float lds[];
    float *Qs = lds + kWaves * 3 * a.s_pad;  // [n_sites][r], shared by the waves
    for (int i = threadIdx.x; i < a.n_sites * a.r; i += kBlock)
        Qs[i] = a.Q[i];
    __syncthreads();
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= a.N)
        return;  // wave-uniform; no workgroup barrier below
    float *al = lds + wave * 3 * a.s_pad, *cq = al + a.s_pad, *ck = cq + a.s_pad;
    const size_t N = (size_t)a.N;
    float ck_sum = 0.0f;
    for (int u = lane; u < a.n_sites; u += kWaveSize) {
        const float *cu = a.coef + u * a.site_stride;
        al[u] = cu[n];
        cq[u] = cu[N + n];
        ck[u] = cu[2 * N + n];
        ck_sum += ck[u];
    }
    ck_sum = wave_sum_t<true>(ck_sum);
    wave_lds_sync();

    // rho of the slot's key: the last r columns of the summary (sliced) or
    // its projected key summary.
    const TK *key = a.sliced ? static_cast<const TK *>(a.Bj) + (size_t)n * a.d + (a.d - a.r)
                             : static_cast<const TK *>(a.KBj) + (size_t)n * a.r;
    float ss = 0.0f;
    for (int e = lane; e < a.r; e += kWaveSize) {
        const float x = load_elem(key + e);
        ss = fmaf(x, x, ss);
    }
    const float rho = sqrtf(wave_sum_t<true>(ss) / (float)a.r + a.eps);
    const float kscale = a.n_sites > 0 ? ck_sum / rho : 0.0f;
    // The key-column term of key element e: sum_t cq_t q_t[e] - kscale * k[e].
    auto key_term = [&](int e) {
        float v = 0.0f;
        for (int u = 0; u < a.n_sites; ++u)
            v = fmaf(cq[u], Qs[u * a.r + e], v);
        return v - kscale * load_elem(key + e);
    };

    const int col = lane * 4;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * 4 < a.d;
    float acc[NCH][4];
    mix_rows<TH, 4, NCH, FULLCOLS>(static_cast<const TH *>(a.dHs) + (size_t)n * a.d + col,
                                   N * a.d, a.n_sites, al, ok, acc);
    TK *prow = static_cast<TK *>(a.dP) + (size_t)n * a.d + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!(FULLCOLS || ok[c]))
            continue;
        if (a.sliced) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int kc = col + c * kWaveSize * 4 + e - (a.d - a.r);
                if (kc >= 0)
                    acc[c][e] += key_term(kc);
            }
        }
        store_raw<TK, 4>(prow + c * kWaveSize * 4, Narrow<TK, 4>::run(acc[c]));
    }
    if (!a.sliced && a.dKP) {
        for (int e = lane; e < a.r; e += kWaveSize)
            store_elem(static_cast<TK *>(a.dKP) + (size_t)n * a.r + e, key_term(e));
    }
}

int check_gather_supported(const BlockGather &g, std::string *why)
{
    if (g.d % 4 != 0 || g.d > 2048) {
        *why = "the block gather needs d % 4 == 0 and d <= 2048";
        return LRAR_EUNSUPPORTED;
    }
    if (g.n_sites > 1024 || g.n_sites * g.r > 16384) {
        *why = "the block gather supports up to 1024 sites and n_sites * r <= 16384";
        return LRAR_EUNSUPPORTED;
    }
    if (g.N > (1 << 30)) {
        *why = "N exceeds 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_block_gather(const BlockGather &g, hipStream_t st, std::string *err)
{
    int rc = check_gather_supported(g, err);
    if (rc)
        return rc;
    if (g.N == 0)
        return LRAR_OK;
    GatherArgs a;
    a.Bj = g.Bj;
    a.KBj = g.KBj;
    a.dHs = g.dHs;
    a.Q = g.Q;
    a.coef = g.coef;
    a.site_stride = g.site_stride;
    a.dP = g.dP;
    a.dKP = g.dKP;
    a.n_sites = (int)g.n_sites;
    a.N = (int)g.N;
    a.d = (int)g.d;
    a.r = (int)g.r;
    a.sliced = g.mode == LRAR_MODE_SLICED ? 1 : 0;
    a.s_pad = (int)((g.n_sites + 3) / 4 * 4);
    a.eps = g.eps;
    const int need = (int)((g.d + 255) / 256);
    int nch = 1;
    while (nch < need)
        nch <<= 1;
    const bool fullcols = g.d % (256 * nch) == 0;
    const size_t lds = ((size_t)kWaves * 3 * a.s_pad + (size_t)a.n_sites * a.r) * sizeof(float);
    const dim3 grid((unsigned)((g.N + kWaves - 1) / kWaves));
    auto go = [&](auto tk, auto th) {
        typedef decltype(tk) TK;
        typedef decltype(th) TH;
        auto launch = [&](auto nchc, auto fc) {
            hipLaunchKernelGGL((block_gather<TK, TH, decltype(nchc)::value, decltype(fc)::value>),
                               grid, dim3(kBlock), lds, st, a);
        };
        auto by_fc = [&](auto nchc) {
            if (fullcols)
                launch(nchc, std::true_type{});
            else
                launch(nchc, std::false_type{});
        };
        switch (nch) {
        case 1: by_fc(std::integral_constant<int, 1>{}); break;
        case 2: by_fc(std::integral_constant<int, 2>{}); break;
        case 4: by_fc(std::integral_constant<int, 4>{}); break;
        default: by_fc(std::integral_constant<int, 8>{}); break;
        }
    };
    if (g.kdtype == LRAR_DTYPE_F32) {
        if (g.dtype == LRAR_DTYPE_BF16)
            go(float{}, uint16_t{});
        else
            go(float{}, float{});
    } else {
        go(uint16_t{}, uint16_t{});  // bf16 sources, bf16 dH
    }
    return hip_status(hipGetLastError(), "block_gather launch", err);
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
    hipError_t e;
    if (p.completed_bf16)  // bf16 completed summaries (bf16 storage only)
        e = launch_block_t<uint16_t, uint16_t>(p, nch, fullcols, lds, nblocks, st);
    else
        e = p.dtype == LRAR_DTYPE_BF16
                ? launch_block_t<uint16_t, float>(p, nch, fullcols, lds, nblocks, st)
                : launch_block_t<float, float>(p, nch, fullcols, lds, nblocks, st);
    return hip_status(e, "block_route_fwd launch", err);
}

}  // namespace lrar
