// Forward kernels of the LR-AttnRes depth routing (Sec. 3.2, Eqs.
// lr_key_norm, lr_attnres_weight, lr_attnres_output) and their launcher.
#include "route_common.h"

namespace lrar {

// ---------------------------------------------------------------------------
// Forward kernels
// ---------------------------------------------------------------------------

// Projected / sliced keys.  Grid: x = token groups of kWaves * TW, y =
// column blocks of NCH*64*VEC (more than one only for very wide rows; each
// column block recomputes the cheap r-dimensional scores).  Wave w owns the
// TW consecutive tokens n0 = (x * kWaves + w) * TW ..: it scores them, takes
// each token's softmax into its own LDS slice, and streams the sources in
// batches of SB, each batch loading the SB sources' rows of all TW tokens
// (adjacent in each source plane) before accumulating them.  Tokens past N
// re-read row N-1 and are not stored; sources past S re-read source S-1
// (the same lines, in flight together) and are not accumulated.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_lr(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
             T *__restrict__ H, int S, int N, int d, int r, int krow, int koff, float eps,
             int s_pad)
{
    constexpr int TW = fwd_tokens_per_wave(NCH);
    constexpr int SB = fwd_sources_per_batch(NCH);
    typedef typename Raw<T, VEC>::type raw_t;
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n0 = ((int)blockIdx.x * kWaves + wave) * TW;
    if (n0 >= N)
        return;  // wave-uniform; this kernel has no workgroup barrier
    const int col = blockIdx.y * (NCH * kWaveSize * VEC) + lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;
    const size_t plane = (size_t)N * d;
    const T *rows[TW];
#pragma unroll
    for (int t = 0; t < TW; ++t)
        rows[t] = V + (size_t)min(n0 + t, N - 1) * d + col;
    float *s = lds + wave * TW * s_pad;

    // One batch is SB sources x TW tokens x NCH column chunks, LPR of whose
    // 16-byte loads are in flight at a time: each group of LPR loads is
    // issued, then accumulated, before the next group goes out.
    constexpr int UNITS = SB * TW * NCH;
    constexpr int LPR = fwd_loads_per_trip(NCH) < UNITS ? fwd_loads_per_trip(NCH) : UNITS;
    raw_t rr[LPR];
    auto load = [&](int i0, int g) {
#pragma unroll
        for (int k = 0; k < LPR; ++k) {
            const int unit = g + k;
            const int u = unit / (TW * NCH), t = (unit / NCH) % TW, c = unit % NCH;
            if (unit < UNITS && (FULLCOLS || ok[c]))
                rr[k] = load_stream<T, VEC, kNtLoad>(rows[t] + (size_t)min(i0 + u, S - 1) * plane +
                                                     c * kWaveSize * VEC);
        }
    };
    float acc[TW][NCH][VEC];
    auto fma = [&](int i0, int g) {
#pragma unroll
        for (int k = 0; k < LPR; ++k) {
            const int unit = g + k;
            const int u = unit / (TW * NCH), t = (unit / NCH) % TW, c = unit % NCH;
            if (unit < UNITS && i0 + u < S && (FULLCOLS || ok[c])) {
                const float a = s[t * s_pad + i0 + u];
                float x[VEC];
                widen(rr[k], x);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[t][c][e] = fmaf(a, x[e], acc[t][c][e]);
            }
        }
    };

    // The first group does not depend on the scores: its loads go out before
    // the key loads, so the two round trips overlap.
    load(0, 0);
    lr_scores_tokens<T, VEC, TW>(keys, q, S, N, r, krow, koff, eps, n0, lane, s, s_pad);
#pragma unroll
    for (int t = 0; t < TW; ++t)
        if (n0 + t < N)
            depth_softmax(s + t * s_pad, s + t * s_pad, S, lane);
#pragma unroll
    for (int t = 0; t < TW; ++t)
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[t][c][e] = 0.0f;
    for (int i0 = 0; i0 < S; i0 += SB) {
#pragma unroll
        for (int g = 0; g < UNITS; g += LPR) {
            if (i0 > 0 || g > 0)
                load(i0, g);
            // The group's loads stay together ahead of their uses.
            __builtin_amdgcn_sched_barrier(0);
            fma(i0, g);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int t = 0; t < TW; ++t)
        if (n0 + t < N)
            store_row<T, VEC, NCH, FULLCOLS>(H + (size_t)(n0 + t) * d + col, ok, acc[t]);
}

// fp32 row segment of VEC values.
template <int VEC>
__device__ __forceinline__ void store_f32(float *p, const float (&x)[VEC])
{
    if constexpr (VEC % 4 == 0) {
#pragma unroll
        for (int k = 0; k < VEC; k += 4)
            *reinterpret_cast<f32x4_t *>(p + k) = f32x4_t{x[k], x[k + 1], x[k + 2], x[k + 3]};
    } else {
#pragma unroll
        for (int k = 0; k < VEC; ++k)
            p[k] = x[k];
    }
}

// The end of a workgroup-split forward: wave w holds the online-softmax
// state (m, l, acc) of its range of one token's sources; the waves publish
// theirs in LDS (stat: 2 kWaves floats; part: the accumulators of waves
// 1..kWaves-1) and wave 0 merges them,
//     m* = max_w m_w,  h = sum_w e^(m_w - m*) acc_w / sum_w e^(m_w - m*) l_w,
// and stores h.  Every wave of the workgroup calls it.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__device__ __forceinline__ void wg_merge_store(float (&acc)[NCH][VEC], float m, float l,
                                               float *stat, float *part, const bool (&ok)[NCH],
                                               T *__restrict__ hrow, int wave, int lane)
{
    constexpr int kRow = NCH * kWaveSize * VEC;
    if (lane == 0) {
        stat[wave] = m;
        stat[kWaves + wave] = l;
    }
    if (wave > 0) {
        float *dst = part + (wave - 1) * kRow + lane * VEC;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
            store_f32<VEC>(dst + c * kWaveSize * VEC, acc[c]);
    }
    __syncthreads();
    if (wave != 0)
        return;
    float mg = stat[0];
#pragma unroll
    for (int u = 1; u < kWaves; ++u)
        mg = fmaxf(mg, stat[u]);
    float scale[kWaves];
    float lsum = 0.0f;
#pragma unroll
    for (int u = 0; u < kWaves; ++u) {
        scale[u] = expf(stat[u] - mg);  // 0 for a wave without sources
        lsum = fmaf(scale[u], stat[kWaves + u], lsum);
    }
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] *= scale[0];
#pragma unroll
        for (int u = 1; u < kWaves; ++u) {
            const float *src = part + (u - 1) * kRow + c * kWaveSize * VEC + lane * VEC;
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[c][e] = fmaf(scale[u], src[e], acc[c][e]);
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] *= inv;
    }
    store_row<T, VEC, NCH, FULLCOLS>(hrow, ok, acc);
}

// The low-rank forward for few tokens: one token per workgroup, its sources
// cut into kWaves consecutive ranges, one per wave.  Each wave keeps the
// online-softmax state of its range (max m_w, sum l_w, accumulator a_w, as
// in route_state_lr) and wave 0 merges the four through LDS (the merge of
// Sec. 3.5 inside one workgroup):
//     m = max_w m_w,  h = sum_w e^(m_w - m) a_w / sum_w e^(m_w - m) l_w.
// Each wave's chain of dependent loads is a quarter as long as in
// route_fwd_lr, which is what bounds a launch with few tokens.  Grid x =
// tokens, y = column blocks; LDS: kWaves * s_pad scores, 2 * kWaves
// statistics, and the accumulators of waves 1..3.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_fwd_lr_wg(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
                T *__restrict__ H, int S, int N, int d, int r, int krow, int koff, float eps,
                int s_pad)
{
    extern __shared__ float lds[];
    constexpr int kRow = NCH * kWaveSize * VEC;  // accumulator floats per wave
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x;
    const int per = (S + kWaves - 1) / kWaves;
    const int i0 = min(S, wave * per);
    const int sc = min(S, i0 + per) - i0;  // 0 for trailing waves when S < 4 per wave
    float *w = lds + wave * s_pad;
    float *stat = lds + kWaves * s_pad;
    float *part = stat + 2 * kWaves;
    const size_t plane = (size_t)N * d;
    const int col = blockIdx.y * kRow + lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        ok[c] = col + c * kWaveSize * VEC < d;
    float acc[NCH][VEC];
    float m = -INFINITY, l = 0.0f;
    if (sc > 0) {  // wave-uniform
        // The first rows of the range do not depend on the scores: their
        // loads go out before the key loads, so the two wait together.
        typedef typename Raw<T, VEC>::type raw_t;
        constexpr int PRE = MixUnroll<NCH>::value;
        const T *vb = V + (size_t)i0 * plane + (size_t)n * d + col;
        raw_t pre[PRE][NCH];
#pragma unroll
        for (int u = 0; u < PRE; ++u)
            if (u < sc)
#pragma unroll
                for (int c = 0; c < NCH; ++c)
                    if (FULLCOLS || ok[c])
                        pre[u][c] = load_stream<T, VEC, kNtLoad>(vb + (size_t)u * plane +
                                                                 c * kWaveSize * VEC);
        lr_scores<T, VEC>(keys + (size_t)i0 * N * krow, q, sc, N, r, krow, koff, eps, n, lane, w,
                          nullptr);
        for (int i = lane; i < sc; i += kWaveSize)
            m = fmaxf(m, w[i]);
        m = wave_max(m);
        for (int i = lane; i < sc; i += kWaveSize) {
            const float e = expf(w[i] - m);
            w[i] = e;
            l += e;
        }
        l = wave_sum(l);
        wave_lds_sync();
        // In source order: the prefetched rows, then the rest of the range.
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[c][e] = 0.0f;
#pragma unroll
        for (int u = 0; u < PRE; ++u) {
            if (u < sc) {
                const float a = w[u];
#pragma unroll
                for (int c = 0; c < NCH; ++c) {
                    if (FULLCOLS || ok[c]) {
                        float x[VEC];
                        widen(pre[u][c], x);
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            acc[c][e] = fmaf(a, x[e], acc[c][e]);
                    }
                }
            }
        }
        if (sc > PRE)
            mix_rows<T, VEC, NCH, FULLCOLS, true>(vb + (size_t)PRE * plane, plane, sc - PRE,
                                                  w + PRE, ok, acc);
    } else {
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[c][e] = 0.0f;
    }
    wg_merge_store<T, VEC, NCH, FULLCOLS>(acc, m, l, stat, part, ok, H + (size_t)n * d + col, wave,
                                          lane);
}

// Online-softmax state of the routing over one chunk of the sources (Sec.
// 3.5, the two-phase form that merges partial routings): chunk c =
// blockIdx.z holds sources c chunk .. min(S, (c + 1) chunk) - 1, and per
// token
//     M = max_i s_i,  L = sum_i exp(s_i - M),  ACC = sum_i exp(s_i - M) o_i,
// so ACC / L is the routing over that chunk, and route_merge combines the
// chunks.  Splitting the sources gives small token counts (decoding) more
// workgroups, and is the step a source-sharded pass exchanges.  Grid x, y
// and layout as route_fwd_lr.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_state_lr(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
               float *__restrict__ M, float *__restrict__ L, float *__restrict__ ACC, int S, int N,
               int d, int r, int krow, int koff, float eps, int s_pad, int chunk)
{
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; this kernel has no workgroup barrier
    const int c = blockIdx.z;
    const int i0 = c * chunk;
    const int sc = min(chunk, S - i0);
    const size_t plane = (size_t)N * d;
    float *w = lds + wave * s_pad;
    lr_scores<T, VEC>(keys + (size_t)i0 * N * krow, q, sc, N, r, krow, koff, eps, n, lane, w,
                      nullptr);
    float m = -INFINITY;
    for (int i = lane; i < sc; i += kWaveSize)
        m = fmaxf(m, w[i]);
    m = wave_max(m);
    float l = 0.0f;
    for (int i = lane; i < sc; i += kWaveSize) {
        const float e = expf(w[i] - m);
        w[i] = e;
        l += e;
    }
    l = wave_sum(l);
    wave_lds_sync();

    const int col = blockIdx.y * (NCH * kWaveSize * VEC) + lane * VEC;
    bool ok[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
        ok[ch] = col + ch * kWaveSize * VEC < d;
    float acc[NCH][VEC];
    mix_rows<T, VEC, NCH, FULLCOLS>(V + (size_t)i0 * plane + (size_t)n * d + col, plane, sc, w, ok,
                                    acc);
    float *arow = ACC + ((size_t)c * N + n) * d + col;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
        if (FULLCOLS || ok[ch])
            store_f32<VEC>(arow + ch * kWaveSize * VEC, acc[ch]);
    if (blockIdx.y == 0 && lane == 0) {
        M[(size_t)c * N + n] = m;
        L[(size_t)c * N + n] = l;
    }
}

// H = (sum_p exp(M_p - m) ACC_p) / (sum_p exp(M_p - m) L_p), m = max_p M_p:
// the routing over the union of the P chunks whose states are given (Sec.
// 3.5's merge).  One wave per token; grid y = column blocks.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__global__ void __launch_bounds__(kBlock)
route_merge(const float *__restrict__ M, const float *__restrict__ L,
            const float *__restrict__ ACC, int P, int N, int d, T *__restrict__ H)
{
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;
    float m = -INFINITY;
    for (int p = lane; p < P; p += kWaveSize)
        m = fmaxf(m, M[(size_t)p * N + n]);
    m = wave_max(m);
    float ls = 0.0f;
    for (int p = lane; p < P; p += kWaveSize)
        ls = fmaf(expf(M[(size_t)p * N + n] - m), L[(size_t)p * N + n], ls);
    ls = wave_sum(ls);
    const int col = blockIdx.y * (NCH * kWaveSize * VEC) + lane * VEC;
    bool ok[NCH];
    float acc[NCH][VEC];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
        ok[ch] = col + ch * kWaveSize * VEC < d;
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[ch][e] = 0.0f;
    }
    for (int p = 0; p < P; ++p) {
        const float wgt = expf(M[(size_t)p * N + n] - m);
        const float *arow = ACC + ((size_t)p * N + n) * d + col;
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            if (FULLCOLS || ok[ch]) {
#pragma unroll
                for (int e = 0; e < VEC; e += (VEC % 4 == 0 ? 4 : 1)) {
                    if constexpr (VEC % 4 == 0) {
                        const f32x4_t x = *reinterpret_cast<const f32x4_t *>(arow + ch * kWaveSize * VEC + e);
                        acc[ch][e] = fmaf(wgt, x.x, acc[ch][e]);
                        acc[ch][e + 1] = fmaf(wgt, x.y, acc[ch][e + 1]);
                        acc[ch][e + 2] = fmaf(wgt, x.z, acc[ch][e + 2]);
                        acc[ch][e + 3] = fmaf(wgt, x.w, acc[ch][e + 3]);
                    } else {
                        acc[ch][e] = fmaf(wgt, arow[ch * kWaveSize * VEC + e], acc[ch][e]);
                    }
                }
            }
        }
    }
    const float inv = 1.0f / ls;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[ch][e] *= inv;
    store_row<T, VEC, NCH, FULLCOLS>(H + (size_t)n * d + col, ok, acc);
}

// Full-rank AttnRes in one pass over the rows: an online softmax over depth.
// Per batch of 4 sources the rows stay in registers while one batched wave
// reduction forms their sum(o^2) and q.o; the running maximum m, the
// normaliser l and the accumulator are rescaled only when m grows.  Reads
// every row once, like the low-rank kernels.
// KIND selects what is written:
//   kFullH     h, one wave per token;
//   kFullState the online-softmax state of chunk c = blockIdx.z (sources
//              c chunk .. min(S, (c + 1) chunk) - 1) to M, L, ACC, as in
//              route_state_lr;
//   kFullWg    h, one token per workgroup (grid x = tokens), its sources
//              cut into kWaves ranges merged by wg_merge_store, as in
//              route_fwd_lr_wg (dynamic LDS: 2 kWaves + (kWaves - 1) row
//              floats).
constexpr int kFullH = 0, kFullState = 1, kFullWg = 2;
template <typename T, int VEC, int NCH, bool FULLCOLS, int KIND = kFullH>
__global__ void __launch_bounds__(kBlock)
route_fwd_full_1p(const T *__restrict__ V, const float *__restrict__ q, T *__restrict__ H,
                  int S, int N, int d, float eps, float *__restrict__ M = nullptr,
                  float *__restrict__ L = nullptr, float *__restrict__ ACC = nullptr, int chunk = 0)
{
    typedef typename Raw<T, VEC>::type raw_t;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = KIND == kFullWg ? (int)blockIdx.x
                  : KIND == kFullH ? xcd_block().x * kWaves + wave
                                   : (int)blockIdx.x * kWaves + wave;
    if (KIND != kFullWg && n >= N)
        return;  // wave-uniform; no workgroup barrier on this path

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
    if constexpr (KIND == kFullState) {
        const int i0 = blockIdx.z * chunk;
        V += (size_t)i0 * plane;
        S = min(chunk, S - i0);
    } else if constexpr (KIND == kFullWg) {
        const int per = (S + kWaves - 1) / kWaves;
        const int i0 = min(S, wave * per);
        V += (size_t)i0 * plane;
        S = min(S, i0 + per) - i0;  // 0 for trailing waves: the loop below is skipped
    }
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
    if constexpr (KIND == kFullWg) {
        extern __shared__ float lds[];
        wg_merge_store<T, VEC, NCH, FULLCOLS>(acc, m, l, lds, lds + 2 * kWaves, ok,
                                              H + (size_t)n * d + col, wave, lane);
        return;
    }
    if constexpr (KIND == kFullState) {
        float *arow = ACC + ((size_t)blockIdx.z * N + n) * d + col;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
            if (FULLCOLS || ok[c])
                store_f32<VEC>(arow + c * kWaveSize * VEC, acc[c]);
        if (lane == 0) {
            M[(size_t)blockIdx.z * N + n] = m;
            L[(size_t)blockIdx.z * N + n] = l;
        }
        return;
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
        if (full && pl.wg_split) {
            hipLaunchKernelGGL((route_fwd_full_1p<T, VEC, NCH, FC, kFullWg>), dim3(pl.nblocks),
                               dim3(kBlock), pl.lds, st, V, p.q, static_cast<T *>(H), (int)p.S,
                               (int)p.N, (int)p.d, p.eps);
        } else if (full) {
            hipLaunchKernelGGL((route_fwd_full_1p<T, VEC, NCH, FC>), dim3(pl.nblocks),
                               dim3(kBlock), 0, st, V, p.q, static_cast<T *>(H), (int)p.S,
                               (int)p.N, (int)p.d, p.eps);
        } else if (pl.wg_split) {
            hipLaunchKernelGGL((route_fwd_lr_wg<T, VEC, NCH, FC>), dim3(pl.nblocks, pl.ysplit),
                               dim3(kBlock), pl.lds, st, V, keys, p.q, static_cast<T *>(H),
                               (int)p.S, (int)p.N, (int)p.d, (int)p.r, krow, koff, p.eps,
                               pl.s_pad);
        } else {
            constexpr int TW = fwd_tokens_per_wave(NCH);
            const int nb = (int)((p.N + kWaves * TW - 1) / (kWaves * TW));
            hipLaunchKernelGGL((route_fwd_lr<T, VEC, NCH, FC>), dim3(nb, pl.ysplit),
                               dim3(kBlock), pl.lds * TW, st, V, keys, p.q, static_cast<T *>(H),
                               (int)p.S, (int)p.N, (int)p.d, (int)p.r, krow, koff, p.eps,
                               pl.s_pad);
        }
        return hipGetLastError();
    });
}

template <typename T, int VEC>
hipError_t launch_state_t(const Problem &p, const Plan &pl, int chunk, float *M, float *L,
                          float *ACC, hipStream_t st)
{
    const T *V = static_cast<const T *>(p.V);
    const T *keys = p.mode == LRAR_MODE_PROJECTED ? static_cast<const T *>(p.K) : V;
    const int krow = p.mode == LRAR_MODE_PROJECTED ? (int)p.r : (int)p.d;
    const int koff = p.mode == LRAR_MODE_SLICED ? (int)(p.d - p.r) : 0;
    const unsigned nchunk = (unsigned)((p.S + chunk - 1) / chunk);
    return dispatch_chunks<VEC>(pl, [&](auto nch, auto fc) -> hipError_t {
        constexpr int NCH = decltype(nch)::value;
        constexpr bool FC = decltype(fc)::value;
        if (p.mode == LRAR_MODE_FULL)
            hipLaunchKernelGGL((route_fwd_full_1p<T, VEC, NCH, FC, kFullState>),
                               dim3(pl.nblocks, 1, nchunk), dim3(kBlock), 0, st, V, p.q,
                               static_cast<T *>(nullptr), (int)p.S, (int)p.N, (int)p.d, p.eps,
                               M, L, ACC, chunk);
        else
            hipLaunchKernelGGL((route_state_lr<T, VEC, NCH, FC>), dim3(pl.nblocks, pl.ysplit, nchunk),
                               dim3(kBlock), pl.lds, st, V, keys, p.q, M, L, ACC, (int)p.S,
                               (int)p.N, (int)p.d, (int)p.r, krow, koff, p.eps, pl.s_pad, chunk);
        return hipGetLastError();
    });
}

template <typename T, int VEC>
hipError_t launch_merge_t(const Plan &pl, const float *M, const float *L, const float *ACC, int P,
                          int N, int d, void *H, hipStream_t st)
{
    return dispatch_chunks<VEC>(pl, [&](auto nch, auto fc) -> hipError_t {
        constexpr int NCH = decltype(nch)::value;
        constexpr bool FC = decltype(fc)::value;
        hipLaunchKernelGGL((route_merge<T, VEC, NCH, FC>), dim3(pl.nblocks, pl.ysplit),
                           dim3(kBlock), 0, st, M, L, ACC, P, N, d, static_cast<T *>(H));
        return hipGetLastError();
    });
}

}  // namespace

int launch_state(const Problem &p, int64_t chunk, float *M, float *L, float *ACC, hipStream_t st,
                 std::string *err)
{
    Problem pc = p;
    pc.S = chunk < p.S ? chunk : p.S;  // the plan of one chunk
    Plan pl;
    if (!make_plan(pc, false, &pl, err))
        return LRAR_EUNSUPPORTED;
    if ((p.S + chunk - 1) / chunk > 65535) {
        *err = "more than 65535 source chunks";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N == 0)
        return LRAR_OK;
    hipError_t e;
    if (p.dtype == LRAR_DTYPE_BF16)
        e = pl.vec > 1 ? launch_state_t<uint16_t, 8>(p, pl, (int)chunk, M, L, ACC, st)
                       : launch_state_t<uint16_t, 1>(p, pl, (int)chunk, M, L, ACC, st);
    else
        e = pl.vec > 1 ? launch_state_t<float, 4>(p, pl, (int)chunk, M, L, ACC, st)
                       : launch_state_t<float, 1>(p, pl, (int)chunk, M, L, ACC, st);
    return hip_status(e, "route_state launch", err);
}

int launch_merge(const float *M, const float *L, const float *ACC, int64_t P, int64_t N, int64_t d,
                 int dtype, void *H, hipStream_t st, std::string *err)
{
    // The column split of a forward over the same rows (the merge has no
    // scores; S only sizes LDS, which the merge does not use).
    Problem pc{nullptr, nullptr, nullptr, 1, N, d, 1, LRAR_MODE_SLICED, dtype, 0.0f, dtype};
    Plan pl;
    if (!make_plan(pc, false, &pl, err))
        return LRAR_EUNSUPPORTED;
    if (P > 1024) {
        *err = "the merge supports at most 1024 states";
        return LRAR_EUNSUPPORTED;
    }
    if (N == 0)
        return LRAR_OK;
    hipError_t e;
    if (dtype == LRAR_DTYPE_BF16)
        e = pl.vec > 1 ? launch_merge_t<uint16_t, 8>(pl, M, L, ACC, (int)P, (int)N, (int)d, H, st)
                       : launch_merge_t<uint16_t, 1>(pl, M, L, ACC, (int)P, (int)N, (int)d, H, st);
    else
        e = pl.vec > 1 ? launch_merge_t<float, 4>(pl, M, L, ACC, (int)P, (int)N, (int)d, H, st)
                       : launch_merge_t<float, 1>(pl, M, L, ACC, (int)P, (int)N, (int)d, H, st);
    return hip_status(e, "route_merge launch", err);
}

int launch_fwd(const Problem &p, void *H, hipStream_t st, std::string *err)
{
    Plan pl;
    if (!make_plan(p, false, &pl, err))
        return LRAR_EUNSUPPORTED;
    if (p.N == 0)
        return LRAR_OK;
    plan_wg_split(p, &pl);
    hipError_t e;
    if (p.dtype == LRAR_DTYPE_BF16)
        e = pl.vec > 1 ? launch_fwd_t<uint16_t, 8>(p, pl, H, st)
                       : launch_fwd_t<uint16_t, 1>(p, pl, H, st);
    else
        e = pl.vec > 1 ? launch_fwd_t<float, 4>(p, pl, H, st) : launch_fwd_t<float, 1>(p, pl, H, st);
    return hip_status(e, "route_fwd launch", err);
}

}  // namespace lrar
