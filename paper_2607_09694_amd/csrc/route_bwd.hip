// Backward kernels of the LR-AttnRes depth routing (the gradient of Sec. 3.2
// Eqs. lr_key_norm, lr_attnres_weight, lr_attnres_output), the fixed-order
// dq reduction, and their launcher.
#include "route_common.h"

#include <mutex>

namespace lrar {

// ---------------------------------------------------------------------------
// Backward kernels (gradient of L = sum_n dH[n] . h[n]; see the header)
// ---------------------------------------------------------------------------

// Key-pass geometry of the projected / sliced backward.  The key pass covers
// `ncols` columns per source: projected keys, the r key columns; sliced keys,
// the value columns from the vector-aligned tail start to d (the tail dV is
// written only here, with the key gradient added).  They are `nkv` vectors of
// KV elements.  A lane owns one vector slot v of one source of a group of
// 64 / LPS sources (LPS = lanes per source, a power of two), so its dq
// partial always belongs to the same columns; rows wider than 64 vectors are
// covered in chunks of 64.
template <int KV> struct KeyChunks { static constexpr int value = KV == 8 ? 1 : KV == 4 ? 2 : 4; };

// Projected / sliced keys.  Each token wave:
//   recomputes s, rho, alpha;  streams the S rows once, forming the partial
//   dots g_i = dH . o_i (one batched reduction per 8 sources) and writing
//   dV_i = alpha_i dH for every column before the key tail;
//   forms ds_i = alpha_i (g_i - sum_l alpha_l g_l);
//   then, lanes over (source, key vector), writes dK (projected) or the last
//   columns of dV including the key gradient (sliced), and accumulates dq.
// dq is reduced per workgroup in a fixed order into partial[blockIdx.x][r].
// T is the storage of V, K, dV and dK; TH that of dH (the same except for
// block sources, whose fp32 summary slots meet the model's bf16 gradient).
// DEFER (block sources, deferred form): only the last source (the block in
// progress) receives gradients, added into the single rows dV [N][d] and
// dK [N][r]; for every other source i the wave writes the three per-token
// coefficients of its gradient instead,
//     coef[i][0][n] = alpha_i,  coef[i][1][n] = ds_i / rho_i,
//     coef[i][2][n] = ds_i s_i / (rho_i r),
// from which dV_i = alpha_i dH + (key columns) coef1 q - coef2 kbar_i.  The
// site's member then retires in the same pass (DeferOut): its gradient is
// the new running row (dO, dK in the model dtype), and it leaves the slot
// (Bp -= o_new, KBp -= k_new) once the slot row has been read for the last
// time (the key columns after the key pass).
// DALL (every source deferred): the coefficients of every source, the last
// one included, are written, and no gradient row at all; each source's
// gradient is then gathered once from the sites that read it (the
// full-source reverse pass).
struct DeferOut {
    float *coef;
    const void *o_new, *k_new;  // model dtype
    void *dO, *dK;              // model dtype
    float *Bp, *KBp;            // the slot of the block in progress
};

template <typename T, typename TH, int VEC, int NCH, bool FULLCOLS, int KV, bool ACC,
          bool DEFER = false, bool DALL = false>
__global__ void __launch_bounds__(kBlock)
route_bwd_lr(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
             const TH *__restrict__ dH, T *__restrict__ dV, T *__restrict__ dK,
             float *__restrict__ partial, int S, int N, int d, int r, int krow, int koff,
             int sliced, int tail_start, float eps, int s_pad, int r_pad, int tpw, int lps,
             DeferOut dfo = DeferOut{})
{
    float *__restrict__ coef = dfo.coef;
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    // wave-uniform (scalar): the stream's buffer descriptors depend on it
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWaveSize);
    float *s = lds + (4 * wave + 0) * s_pad;
    float *rho = lds + (4 * wave + 1) * s_pad;
    float *alpha = lds + (4 * wave + 2) * s_pad;
    float *g = lds + (4 * wave + 3) * s_pad;
    float *stage = lds + 4 * kWaves * s_pad;  // [kWaves][r_pad]

    constexpr int KC = KeyChunks<KV>::value;
    const int kbase = sliced ? tail_start : 0;   // first column of the key pass
    const int kshift = sliced ? d - r : 0;       // column of key element 0
    const int nkv = (sliced ? d - tail_start : r) / KV;
    const int isub = lane / lps;                 // source within a group
    const int spi = kWaveSize / lps;             // sources per group
    const int vl = lane % lps;
    const float inv_r = 1.0f / (float)r;

    // Per-lane key-pass constants: q at the lane's key columns.
    float qk[KC][KV], dq_acc[KC][KV];
#pragma unroll
    for (int k = 0; k < KC; ++k)
#pragma unroll
        for (int e = 0; e < KV; ++e) {
            const int v = k * kWaveSize + vl;
            const int j = kbase + v * KV + e - kshift;
            qk[k][e] = (v < nkv && j >= 0) ? q[j] : 0.0f;
            dq_acc[k][e] = 0.0f;
        }

    const int col = lane * VEC;
    bool ok[NCH], wr[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        ok[c] = col + c * kWaveSize * VEC < d;
        wr[c] = col + c * kWaveSize * VEC < tail_start;
    }
    const size_t plane = (size_t)N * d;

    const int bx = blockIdx.x;
    for (int t = 0; t < tpw; ++t) {
        const int n = (bx * tpw + t) * kWaves + wave;
        if (n >= N)
            break;  // wave-uniform; the workgroup barrier below is outside the loop
        lr_scores<T, VEC, std::is_same<T, float>::value>(keys, q, S, N, r, krow, koff, eps, n,
                                                          lane, s, rho);
        depth_softmax<std::is_same<T, float>::value>(s, alpha, S, lane);

        typedef typename Raw<T, VEC>::type raw_t;
        float dh[NCH][VEC];
        const TH *dhrow = dH + (size_t)n * d + col;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (FULLCOLS || ok[c]) {
                widen(load_raw<TH, VEC>(dhrow + c * kWaveSize * VEC), dh[c]);
            } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    dh[c][e] = 0.0f;
            }
        }
        const T *vbase = V + (size_t)n * d + col;
        T *dvbase = dV + (size_t)n * d + col;
        constexpr int L = BwdInflight<NCH>::value;
        // With 16-byte vectors every access of the stream goes through a
        // per-row buffer resource: source i's value row (no bytes past the
        // last source) and its gradient row (bytes up to the key tail, none
        // when the source takes no gradient row here).  Lanes past the row
        // end and sources past S read zeros and store nothing, with no branch
        // around any access, so the compiler's wait counts let the stores and
        // the next loads stay in flight.  Scalar rows keep guarded accesses.
        constexpr bool BUF = VEC > 1;
        for (int i0 = 0; i0 < S; i0 += 8) {
            float part[8];
#pragma unroll
            for (int h = 0; h < 8; h += L) {
                raw_t raw[L][NCH], old[ACC ? L : 1][NCH];
                __amdgpu_buffer_rsrc_t rv[L], rd[L];
#pragma unroll
                for (int u = 0; u < L; ++u) {
                    const int i = i0 + h + u;
                    const bool live = i < S;
                    const bool takes = live && (!DEFER || (!DALL && i == S - 1));
                    if constexpr (BUF) {
                        const size_t ic = (size_t)min(i, S - 1);  // in-range base
                        rv[u] = row_rsrc(V + (ic * N + n) * d, live ? d * (int)sizeof(T) : 0);
                        // every source of a fully deferred step takes no row (dV may be NULL)
                        rd[u] = row_rsrc(DALL ? nullptr : dV + (DEFER ? (size_t)n : ic * N + n) * d,
                                         takes ? tail_start * (int)sizeof(T) : 0);
#pragma unroll
                        for (int c = 0; c < NCH; ++c) {
                            const int off = (col + c * kWaveSize * VEC) * (int)sizeof(T);
                            raw[u][c] = buffer_load16<T, VEC, kBwdNtLoad>(rv[u], off);
                            if constexpr (ACC)
                                old[u][c] = buffer_load16<T, VEC, kBwdNtLoad>(rd[u], off);
                        }
                    } else if (live) {
#pragma unroll
                        for (int c = 0; c < NCH; ++c)
                            if (FULLCOLS || ok[c]) {
                                const size_t off = (size_t)i * plane + c * kWaveSize * VEC;
                                raw[u][c] = load_stream<T, VEC, kNtLoad>(vbase + off);
                                if constexpr (ACC)
                                    if (wr[c] && takes)
                                        old[u][c] = load_stream<T, VEC, kNtLoad>(
                                            dvbase + (DEFER ? c * kWaveSize * VEC : off));
                            }
                    }
                }
#pragma unroll
                for (int u = 0; u < L; ++u) {
                    float p = 0.0f;
                    const int i = i0 + h + u;
                    if (BUF || i < S) {
                        const float a = i < S ? alpha[min(i, S - 1)] : 0.0f;
#pragma unroll
                        for (int c = 0; c < NCH; ++c) {
                            if (BUF || FULLCOLS || ok[c]) {
                                float x[VEC], y[VEC];
                                widen(raw[u][c], x);
#pragma unroll
                                for (int e = 0; e < VEC; ++e) {
                                    p = fmaf(dh[c][e], x[e], p);
                                    y[e] = a * dh[c][e];
                                }
                                const bool wdv = wr[c] && i < S && (!DEFER || (!DALL && i == S - 1));
                                if constexpr (BUF) {
                                    if constexpr (ACC)
                                        add_stored(y, old[u][c]);
                                    buffer_store16<T, VEC, kBwdNtStore>(
                                        rd[u], (col + c * kWaveSize * VEC) * (int)sizeof(T),
                                        Narrow<T, VEC>::run(y));
                                } else {
                                    if constexpr (ACC)
                                        if (wdv)
                                            add_stored(y, old[u][c]);
                                    if (wdv)
                                        store_stream<T, VEC, kNtStore>(
                                            dvbase + (DEFER ? 0 : (size_t)i * plane) + c * kWaveSize * VEC,
                                            Narrow<T, VEC>::run(y));
                                }
                                if constexpr (DEFER && !DALL) {
                                    if (wdv) {
                                        // retire: dO = the new running row;
                                        // the member leaves the slot
                                        const size_t ro = (size_t)n * d + col + c * kWaveSize * VEC;
                                        store_stream<TH, VEC, kNtStore>(
                                            static_cast<TH *>(dfo.dO) + ro, Narrow<TH, VEC>::run(y));
                                        float o[VEC];
                                        widen(load_raw<TH, VEC>(static_cast<const TH *>(dfo.o_new) + ro), o);
#pragma unroll
                                        for (int e = 0; e < VEC; ++e)
                                            x[e] -= o[e];
                                        store_raw<float, VEC>(dfo.Bp + ro, Narrow<float, VEC>::run(x));
                                    }
                                }
                            }
                        }
                    }
                    part[h + u] = p;
                }
                // One step of L sources at a time: the dots of this step are
                // formed before the next step's loads go out, so at most one
                // step's rows are in flight per wave.
#pragma unroll
                for (int u = 0; u < L; ++u)
                    asm volatile("" : "+v"(part[h + u])::"memory");
            }
            const float tot = multi_sum<8>(part, lane);
            const int idx = multi_sum_index<8>(lane);
            if (multi_sum_writer<8>(lane) && i0 + idx < S)
                g[i0 + idx] = tot;
        }
        wave_lds_sync();
        float gb = 0.0f;
        for (int i = lane; i < S; i += kWaveSize)
            gb = fmaf(alpha[i], g[i], gb);
        gb = wave_sum_t<std::is_same<T, float>::value>(gb);
        for (int i = lane; i < S; i += kWaveSize)
            g[i] = alpha[i] * (g[i] - gb);  // g now holds ds
        wave_lds_sync();

        // Key pass: lanes over (source, key vector).
#pragma unroll
        for (int k = 0; k < KC; ++k) {
            const int v = k * kWaveSize + vl;
            if (k * kWaveSize >= nkv)
                break;  // wave-uniform
            const bool vok = v < nkv;
            const int c0 = kbase + v * KV;  // projected: key index; sliced: value column
            float dhk[KV];
            if (sliced && vok) {
                widen(load_raw<TH, KV>(dH + (size_t)n * d + c0), dhk);
            } else {
#pragma unroll
                for (int e = 0; e < KV; ++e)
                    dhk[e] = 0.0f;
            }
#pragma unroll 4
            for (int i0 = 0; i0 < S; i0 += spi) {
                const int i = i0 + isub;
                if (!vok || i >= S)
                    continue;
                const size_t row = (size_t)i * N + n;
                const float ri = 1.0f / rho[i];
                const float dsi = g[i];
                const float cq = dsi * ri;              // ds_i / rho_i
                const float ck = cq * s[i] * inv_r;     // ds_i s_i / (rho_i r)
                const bool defer_i = DEFER && (DALL || i < S - 1);
                const size_t orow = DEFER ? (size_t)n : row;  // output row of source i
                if (defer_i && k == 0 && vl == 0) {
                    coef[((size_t)i * 3 + 0) * N + n] = alpha[i];
                    coef[((size_t)i * 3 + 1) * N + n] = cq;
                    coef[((size_t)i * 3 + 2) * N + n] = ck;
                }
                float x[KV], y[KV];
                if (!sliced) {
                    widen(load_raw<T, KV>(keys + row * krow + c0), x);
#pragma unroll
                    for (int e = 0; e < KV; ++e) {
                        const float kb = x[e] * ri;
                        y[e] = fmaf(cq, qk[k][e], -ck * kb);
                        dq_acc[k][e] = fmaf(dsi, kb, dq_acc[k][e]);
                    }
                    if (defer_i)
                        continue;
                    if constexpr (ACC)
                        add_stored(y, load_raw<T, KV>(dK + orow * r + c0));
                    store_raw<T, KV>(dK + orow * r + c0, Narrow<T, KV>::run(y));
                    if constexpr (DEFER && !DALL) {
                        // retire the member's key: dK = the new running key
                        // row; the key leaves the slot's key summary
                        const size_t ro = (size_t)n * r + c0;
#pragma unroll
                        for (int e = 0; e < KV; ++e) {
                            store_elem(static_cast<TH *>(dfo.dK) + ro + e, y[e]);
                            dfo.KBp[ro + e] =
                                x[e] - load_elem(static_cast<const TH *>(dfo.k_new) + ro + e);
                        }
                    }
                } else {
                    widen(load_raw<T, KV>(V + row * d + c0), x);
                    const float a = alpha[i];
#pragma unroll
                    for (int e = 0; e < KV; ++e) {
                        y[e] = a * dhk[e];
                        if (c0 + e >= kshift) {
                            const float kb = x[e] * ri;
                            y[e] += fmaf(cq, qk[k][e], -ck * kb);
                            dq_acc[k][e] = fmaf(dsi, kb, dq_acc[k][e]);
                        }
                    }
                    if (defer_i)
                        continue;
                    if constexpr (ACC)
                        add_stored(y, load_raw<T, KV>(dV + orow * d + c0));
                    store_raw<T, KV>(dV + orow * d + c0, Narrow<T, KV>::run(y));
                    if constexpr (DEFER && !DALL) {
                        // retire the member's columns of the key pass: its
                        // gradient, and the slot without it (the slot row
                        // was read here for the last time)
                        const size_t ro = (size_t)n * d + c0;
#pragma unroll
                        for (int e = 0; e < KV; ++e) {
                            store_elem(static_cast<TH *>(dfo.dO) + ro + e, y[e]);
                            dfo.Bp[ro + e] =
                                x[e] - load_elem(static_cast<const TH *>(dfo.o_new) + ro + e);
                        }
                    }
                }
            }
        }
        wave_lds_sync();  // LDS of this token is reused by the next one
    }

    // Fixed-order reduction of dq: over the source groups of the wave
    // (butterfly over the lane bits above the vector slot), then over the
    // waves of the workgroup in wave order.
#pragma unroll
    for (int k = 0; k < KC; ++k)
#pragma unroll
        for (int e = 0; e < KV; ++e)
            for (int m = lps; m < kWaveSize; m <<= 1)
                dq_acc[k][e] += __shfl_xor(dq_acc[k][e], m, kWaveSize);
    float *my = stage + wave * r_pad;
    for (int j = lane; j < r; j += kWaveSize)
        my[j] = 0.0f;
    wave_lds_sync();
    if (isub == 0) {
#pragma unroll
        for (int k = 0; k < KC; ++k) {
            const int v = k * kWaveSize + vl;
            if (v < nkv) {
#pragma unroll
                for (int e = 0; e < KV; ++e) {
                    const int j = kbase + v * KV + e - kshift;
                    if (j >= 0)
                        my[j] = dq_acc[k][e];
                }
            }
        }
    }
    __syncthreads();
    for (int j = threadIdx.x; j < r; j += kBlock) {
        float sum = 0.0f;
        for (int w = 0; w < kWaves; ++w)
            sum += stage[w * r_pad + j];
        partial[(size_t)bx * r + j] = sum;
    }
}

// Full-rank AttnRes backward: pass 1 reads the rows once for sum(o^2), q.o
// and dH.o (one batched reduction per 4 sources); pass 2 re-reads them to
// write dV_i = alpha_i dH + (ds_i/rho_i)(q - o_i s_i/(rho_i d)) and to
// accumulate dq = sum ds_i o_i / rho_i per lane column.
template <typename T, int VEC, int NCH, bool FULLCOLS, bool ACC>
__global__ void __launch_bounds__(kBlock)
route_bwd_full(const T *__restrict__ V, const float *__restrict__ q, const T *__restrict__ dH,
               T *__restrict__ dV, float *__restrict__ partial, int S, int N, int d, float eps,
               int s_pad, int tpw)
{
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    float *ss = lds + (4 * wave + 0) * s_pad;     // sum o^2, then rho
    float *sc = lds + (4 * wave + 1) * s_pad;     // q.o, then the score
    float *g = lds + (4 * wave + 2) * s_pad;      // dH.o, then ds
    float *alpha = lds + (4 * wave + 3) * s_pad;
    float *stage = lds + 4 * kWaves * s_pad;      // [d]

    const int col = lane * VEC;
    bool ok[NCH];
    float qv[NCH][VEC], dqa[NCH][VEC];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        ok[c] = col + c * kWaveSize * VEC < d;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            qv[c][e] = (FULLCOLS || ok[c]) ? q[col + c * kWaveSize * VEC + e] : 0.0f;
            dqa[c][e] = 0.0f;
        }
    }
    const size_t plane = (size_t)N * d;
    const float inv_d = 1.0f / (float)d;

    const int bx = blockIdx.x;
    for (int t = 0; t < tpw; ++t) {
        const int n = (bx * tpw + t) * kWaves + wave;
        if (n >= N)
            break;  // wave-uniform; the workgroup barriers are after the loop
        float dh[NCH][VEC];
        const T *vbase = V + (size_t)n * d + col;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (FULLCOLS || ok[c]) {
                widen(load_raw<T, VEC>(dH + (size_t)n * d + col + c * kWaveSize * VEC), dh[c]);
            } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    dh[c][e] = 0.0f;
            }
        }
        for (int i0 = 0; i0 < S; i0 += 4) {
            float part[16];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                float a = 0.0f, b = 0.0f, p = 0.0f;
                if (i0 + u < S) {
#pragma unroll
                    for (int c = 0; c < NCH; ++c) {
                        if (FULLCOLS || ok[c]) {
                            float x[VEC];
                            widen(load_raw<T, VEC>(vbase + (size_t)(i0 + u) * plane +
                                                   c * kWaveSize * VEC), x);
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                a = fmaf(x[e], x[e], a);
                                b = fmaf(qv[c][e], x[e], b);
                                p = fmaf(dh[c][e], x[e], p);
                            }
                        }
                    }
                }
                part[u] = a;
                part[4 + u] = b;
                part[8 + u] = p;
                part[12 + u] = 0.0f;
            }
            const float tot = multi_sum<16>(part, lane);
            const int idx = multi_sum_index<16>(lane);
            const int i = i0 + (idx & 3);
            if (multi_sum_writer<16>(lane) && idx < 12 && i < S)
                (idx < 4 ? ss : idx < 8 ? sc : g)[i] = tot;
        }
        wave_lds_sync();
        for (int i = lane; i < S; i += kWaveSize) {
            const float rho = sqrtf(ss[i] / (float)d + eps);
            ss[i] = rho;
            sc[i] = sc[i] / rho;
        }
        depth_softmax(sc, alpha, S, lane);
        float gb = 0.0f;
        for (int i = lane; i < S; i += kWaveSize)
            gb = fmaf(alpha[i], g[i], gb);
        gb = wave_sum(gb);
        for (int i = lane; i < S; i += kWaveSize)
            g[i] = alpha[i] * (g[i] - gb);
        wave_lds_sync();

        T *dvbase = dV + (size_t)n * d + col;
        for (int i = 0; i < S; ++i) {
            const float a = alpha[i];
            const float c1 = g[i] / ss[i];                  // ds_i / rho_i
            const float c2 = c1 * sc[i] / ss[i] * inv_d;    // ds_i s_i / (rho_i^2 d)
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULLCOLS || ok[c]) {
                    float x[VEC], y[VEC];
                    widen(load_raw<T, VEC>(vbase + (size_t)i * plane + c * kWaveSize * VEC), x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        y[e] = fmaf(a, dh[c][e], fmaf(c1, qv[c][e], -c2 * x[e]));
                        dqa[c][e] = fmaf(c1, x[e], dqa[c][e]);
                    }
                    if constexpr (ACC)
                        add_stored(y, load_raw<T, VEC>(dvbase + (size_t)i * plane +
                                                       c * kWaveSize * VEC));
                    store_raw<T, VEC>(dvbase + (size_t)i * plane + c * kWaveSize * VEC,
                                      Narrow<T, VEC>::run(y));
                }
            }
        }
        wave_lds_sync();
    }

    // Fixed-order workgroup reduction of dq: waves add their columns in turn.
    for (int w = 0; w < kWaves; ++w) {
        if (wave == w) {
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULLCOLS || ok[c]) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        float *p = stage + col + c * kWaveSize * VEC + e;
                        *p = (w == 0 ? 0.0f : *p) + dqa[c][e];
                    }
                }
            }
        }
        __syncthreads();
    }
    for (int j = threadIdx.x; j < d; j += kBlock)
        partial[(size_t)bx * d + j] = stage[j];
}

// dq[j] = sum_b partial[b][j] in a fixed order: one workgroup per column;
// thread t sums rows t, t+256, ... in order, then a fixed pairwise tree over
// the 256 thread sums.  Writes zeros when nblocks = 0.
template <bool ACC>
__global__ void __launch_bounds__(256)
dq_reduce(const float *__restrict__ partial, float *__restrict__ dq, int nblocks, int ncols)
{
    __shared__ float red[256];
    const int t = threadIdx.x;
    const int j = blockIdx.x;
    float s = 0.0f;
    for (int b = t; b < nblocks; b += 256)
        s += partial[(size_t)b * ncols + j];
    red[t] = s;
    __syncthreads();
#pragma unroll
    for (int w = 128; w >= 1; w >>= 1) {
        if (t < w)
            red[t] += red[t + w];
        __syncthreads();
    }
    if (t == 0)
        dq[j] = ACC ? dq[j] + red[0] : red[0];
}

hipError_t launch_dq_reduce(const float *partial, float *dq, int nblocks, int ncols,
                            bool accumulate, hipStream_t st)
{
    if (accumulate)
        hipLaunchKernelGGL(dq_reduce<true>, dim3(ncols), dim3(256), 0, st, partial, dq, nblocks,
                           ncols);
    else
        hipLaunchKernelGGL(dq_reduce<false>, dim3(ncols), dim3(256), 0, st, partial, dq, nblocks,
                           ncols);
    return hipGetLastError();
}

namespace {

// Key-pass vector width and lanes per source of the projected / sliced
// backward: 16-byte vectors when the key rows allow it, else scalars.
struct KeyPass {
    int kv, lps, nkv;
};

KeyPass key_pass(const Problem &p, const Plan &pl)
{
    const bool sliced = p.mode == LRAR_MODE_SLICED;
    const int tail_start = sliced ? (int)((p.d - p.r) / pl.vec * pl.vec) : (int)p.d;
    KeyPass k;
    k.kv = pl.vec > 1 && (sliced || p.r % pl.vec == 0) ? pl.vec : 1;
    k.nkv = (int)(sliced ? p.d - tail_start : p.r) / k.kv;
    k.lps = 1;
    while (k.lps < k.nkv && k.lps < kWaveSize)
        k.lps <<= 1;
    return k;
}

template <typename T, typename TH, int VEC, bool ACC, bool DEFER = false, bool DALL = false>
hipError_t launch_bwd_t(const Problem &p, const Plan &pl, const void *dH, void *dV, void *dK,
                        float *partial, hipStream_t st, const DeferOut &dfo = DeferOut{})
{
    const T *V = static_cast<const T *>(p.V);
    const int tail_start = p.mode == LRAR_MODE_SLICED ? (int)((p.d - p.r) / pl.vec * pl.vec)
                                                      : (int)p.d;
    const T *keys = p.mode == LRAR_MODE_PROJECTED ? static_cast<const T *>(p.K) : V;
    const int krow = p.mode == LRAR_MODE_PROJECTED ? (int)p.r : (int)p.d;
    const int koff = p.mode == LRAR_MODE_SLICED ? (int)(p.d - p.r) : 0;
    const KeyPass kp = key_pass(p, pl);
    return dispatch_chunks<VEC>(pl, [&](auto nch, auto fc) -> hipError_t {
        constexpr int NCH = decltype(nch)::value;
        constexpr bool FC = decltype(fc)::value;
        if constexpr (std::is_same<T, TH>::value && !DEFER) {
            if (p.mode == LRAR_MODE_FULL) {
                hipLaunchKernelGGL((route_bwd_full<T, VEC, NCH, FC, ACC>), dim3(pl.nblocks),
                                   dim3(kBlock), pl.lds, st, V, p.q, static_cast<const T *>(dH),
                                   static_cast<T *>(dV), partial, (int)p.S, (int)p.N, (int)p.d,
                                   p.eps, pl.s_pad, pl.tpw);
                return hipGetLastError();
            }
        }
        auto launch = [&](auto kvc) {
            constexpr int KV = decltype(kvc)::value;
            hipLaunchKernelGGL((route_bwd_lr<T, TH, VEC, NCH, FC, KV, ACC, DEFER, DALL>),
                               dim3(pl.nblocks), dim3(kBlock), pl.lds, st, V, keys, p.q,
                               static_cast<const TH *>(dH), static_cast<T *>(dV),
                               static_cast<T *>(dK), partial, (int)p.S, (int)p.N, (int)p.d,
                               (int)p.r, krow, koff, p.mode == LRAR_MODE_SLICED ? 1 : 0,
                               tail_start, p.eps, pl.s_pad, pl.r_pad, pl.tpw, kp.lps, dfo);
        };
        if constexpr (VEC > 1) {
            if (kp.kv == VEC)
                launch(std::integral_constant<int, VEC>{});
            else
                launch(std::integral_constant<int, 1>{});
        } else {
            launch(std::integral_constant<int, 1>{});
        }
        return hipGetLastError();
    });
}

// The routing backward (accumulating dV / dK when ACC) and the dq reduction
// (accumulating when ACCQ).  Mixed storage (fp32 values, bf16 dH) exists only
// for the accumulating form used by block sources.
template <bool ACC, bool ACCQ>
hipError_t launch_bwd_acc(const Problem &p, const Plan &pl, const void *dH, void *dV, void *dK,
                          float *dq, float *partial, hipStream_t st)
{
    hipError_t e = hipSuccess;
    if (p.N > 0) {
        const bool mixed = p.dtype == LRAR_DTYPE_F32 && p.dh_dtype == LRAR_DTYPE_BF16;
        if (p.dtype == LRAR_DTYPE_BF16)
            e = pl.vec > 1 ? launch_bwd_t<uint16_t, uint16_t, 8, ACC>(p, pl, dH, dV, dK, partial, st)
                           : launch_bwd_t<uint16_t, uint16_t, 1, ACC>(p, pl, dH, dV, dK, partial, st);
        else if (!mixed)
            e = pl.vec > 1 ? launch_bwd_t<float, float, 4, ACC>(p, pl, dH, dV, dK, partial, st)
                           : launch_bwd_t<float, float, 1, ACC>(p, pl, dH, dV, dK, partial, st);
        else if constexpr (ACC)
            e = pl.vec > 1 ? launch_bwd_t<float, uint16_t, 4, ACC>(p, pl, dH, dV, dK, partial, st)
                           : launch_bwd_t<float, uint16_t, 1, ACC>(p, pl, dH, dV, dK, partial, st);
        else
            e = hipErrorInvalidValue;
        if (e != hipSuccess)
            return e;
    }
    const int ncols = (int)(p.mode == LRAR_MODE_FULL ? p.d : p.r);
    const int nb = p.N > 0 ? pl.nblocks : 0;
    hipLaunchKernelGGL(dq_reduce<ACCQ>, dim3(ncols), dim3(256), 0, st, partial, dq, nb, ncols);
    return hipGetLastError();
}

}  // namespace

int launch_bwd(const Problem &p, const void *dH, void *dV, void *dK, float *dq, void *ws,
               bool accumulate, hipStream_t st, std::string *err)
{
    Plan pl;
    if (!make_plan(p, true, &pl, err))
        return LRAR_EUNSUPPORTED;
    float *partial = static_cast<float *>(ws);
    const hipError_t e =
        accumulate ? launch_bwd_acc<true, true>(p, pl, dH, dV, dK, dq, partial, st)
                   : launch_bwd_acc<false, false>(p, pl, dH, dV, dK, dq, partial, st);
    return hip_status(e, "route_bwd launch", err);
}

// Block sources, one site of the reverse pass: accumulate the slot gradients
// (fp32) from the model-dtype dH, write dq, then retire the site (the
// member's gradient is its slot's gradient so far; the member leaves its
// slot).
int launch_block_bwd_deferred(const Problem &p, const BlockRetire &br, const void *dH, float *dP,
                              float *dKP, float *coef, float *dq, void *ws, hipStream_t st,
                              std::string *err)
{
    Plan pl;
    if (!make_plan(p, true, &pl, err))
        return LRAR_EUNSUPPORTED;
    float *partial = static_cast<float *>(ws);
    // The retire step runs inside the backward kernel (DeferOut).
    const size_t plane = (size_t)p.N * p.d, kplane = (size_t)p.N * p.r;
    DeferOut dfo;
    dfo.coef = coef;
    dfo.o_new = br.o_new;
    dfo.k_new = br.k_new;
    dfo.dO = br.dO;
    dfo.dK = br.dK;
    dfo.Bp = br.B + br.j * plane;
    dfo.KBp = br.KB ? br.KB + br.j * kplane : nullptr;
    hipError_t e = hipSuccess;
    if (p.N > 0) {
        if (p.dh_dtype == LRAR_DTYPE_BF16)
            e = pl.vec > 1
                    ? launch_bwd_t<float, uint16_t, 4, true, true>(p, pl, dH, dP, dKP, partial, st, dfo)
                    : launch_bwd_t<float, uint16_t, 1, true, true>(p, pl, dH, dP, dKP, partial, st, dfo);
        else
            e = pl.vec > 1
                    ? launch_bwd_t<float, float, 4, true, true>(p, pl, dH, dP, dKP, partial, st, dfo)
                    : launch_bwd_t<float, float, 1, true, true>(p, pl, dH, dP, dKP, partial, st, dfo);
    }
    if (e == hipSuccess) {
        const int ncols = (int)p.r;
        hipLaunchKernelGGL(dq_reduce<false>, dim3(ncols), dim3(256), 0, st, partial, dq,
                           p.N > 0 ? pl.nblocks : 0, ncols);
        e = hipGetLastError();
    }
    return hip_status(e, "block_route_bwd_deferred launch", err);
}

int launch_bwd_deferred_all(const Problem &p, const void *dH, float *coef, float *dq, void *ws,
                            hipStream_t st, std::string *err)
{
    if (p.mode == LRAR_MODE_FULL) {
        *err = "the deferred backward takes projected or sliced keys";
        return LRAR_EUNSUPPORTED;
    }
    Plan pl;
    if (!make_plan(p, true, &pl, err))
        return LRAR_EUNSUPPORTED;
    float *partial = static_cast<float *>(ws);
    DeferOut dfo;
    dfo.coef = coef;
    hipError_t e = hipSuccess;
    if (p.N > 0) {
        if (p.dtype == LRAR_DTYPE_BF16)
            e = pl.vec > 1 ? launch_bwd_t<uint16_t, uint16_t, 8, false, true, true>(
                                 p, pl, dH, nullptr, nullptr, partial, st, dfo)
                           : launch_bwd_t<uint16_t, uint16_t, 1, false, true, true>(
                                 p, pl, dH, nullptr, nullptr, partial, st, dfo);
        else
            e = pl.vec > 1 ? launch_bwd_t<float, float, 4, false, true, true>(
                                 p, pl, dH, nullptr, nullptr, partial, st, dfo)
                           : launch_bwd_t<float, float, 1, false, true, true>(
                                 p, pl, dH, nullptr, nullptr, partial, st, dfo);
    }
    if (e == hipSuccess)
        e = launch_dq_reduce(partial, dq, p.N > 0 ? pl.nblocks : 0, (int)p.r, false, st);
    return hip_status(e, "route_bwd_deferred launch", err);
}

int launch_block_bwd(const Problem &p, const BlockRetire &br, const void *dH, void *dB,
                     void *dKB, float *dq, void *ws, hipStream_t st, std::string *err)
{
    Plan pl;
    if (!make_plan(p, true, &pl, err))
        return LRAR_EUNSUPPORTED;
    hipError_t e = launch_bwd_acc<true, false>(p, pl, dH, dB, dKB, dq, static_cast<float *>(ws),
                                               st);
    if (e == hipSuccess && p.N > 0)
        e = launch_block_retire(br, st);
    return hip_status(e, "block_route_bwd launch", err);
}

// ---------------------------------------------------------------------------
// Allocation-free backward: the dq partials in a file-scope device array
// ---------------------------------------------------------------------------

// The per-workgroup dq partials of lr_attnres_route_bwd_noalloc live here
// instead of in a caller workspace.  Every device the library runs on holds
// its own copy until the process ends; all calls on one device share it, and
// each launch overwrites the rows it later reads, so nothing has to start at
// zero.  Host code never passes this name to a kernel: it stands for a host
// shadow, and the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
float *g_scratch_addr[kMaxDevices];

// Device address of `scratch` on device `dev`, looked up once per device
// with that device current.
int scratch_address(int dev, float **out, std::string *err)
{
    if (dev < 0 || dev >= kMaxDevices) {
        *err = "device index " + std::to_string(dev) + " beyond the allocation-free backward's " +
               std::to_string(kMaxDevices) + " devices";
        return LRAR_EUNSUPPORTED;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_addr[dev]) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e != hipSuccess)
            return hip_status(e, "hipGetDevice", err);
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess)
            return hip_status(e, "hipSetDevice", err);
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t back = hipSetDevice(cur);
            if (e == hipSuccess)
                e = back;
        }
        if (e != hipSuccess)
            return hip_status(e, "hipGetSymbolAddress(scratch)", err);
        g_scratch_addr[dev] = static_cast<float *>(p);
    }
    *out = g_scratch_addr[dev];
    return LRAR_OK;
}

}  // namespace

int launch_bwd_noalloc(const Problem &p, const void *dH, void *dV, void *dK, float *dq,
                       hipStream_t st, std::string *err)
{
    const size_t need = bwd_workspace_bytes(p);
    if (need > kNoAllocScratchBytes) {
        *err = "the allocation-free backward needs " + std::to_string(need) +
               " bytes of dq partials; its device array holds " +
               std::to_string(kNoAllocScratchBytes);
        return LRAR_EUNSUPPORTED;
    }
    int dev = -1;
    hipError_t e = st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_status(e, st ? "hipStreamGetDevice" : "hipGetDevice", err);
    float *ws = nullptr;
    const int rc = scratch_address(dev, &ws, err);
    if (rc != LRAR_OK)
        return rc;
    return launch_bwd(p, dH, dV, dK, dq, ws, false, st, err);
}

}  // namespace lrar
