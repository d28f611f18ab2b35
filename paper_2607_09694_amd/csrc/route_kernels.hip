// gfx950 kernels of the LR-AttnRes depth routing (arXiv 2607.09694, Sec. 3)
// and their host-side launchers.
//
// Work decomposition: one wave64 owns one token n ("token wave"); a
// workgroup is kWaves token waves on consecutive tokens, so the projected
// keys of neighbouring tokens, which share cache lines, are read together.
// Per token the wave
//   1. scores the S sources from their keys, lane = source (P-LR / S-LR),
//   2. takes the softmax over depth with wave reductions, keeping the weights
//      in a wave-private LDS slice (never written to HBM),
//   3. streams the S value rows of the token through the wave: each lane
//      owns NCH 16-byte column vectors of the row, widens bf16 to fp32 and
//      accumulates with fp32 FMAs; the rows are independent 2-8 KB contiguous
//      reads, several sources in flight per lane.
// Full-rank AttnRes (the key is the whole value) scores each source with a
// wave-wide dot product instead, folded into the same single stream of the
// rows by an online softmax.
// The work is a bandwidth-bound gather-reduce (about one flop per byte), so
// it uses no MFMA: the roofline is HBM.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string>
#include <type_traits>

#include "route_device.h"
#include "route_launch.h"

namespace lrar {

constexpr int kWaves = 4;                    // token waves per workgroup
constexpr int kBlock = kWaves * kWaveSize;   // 256 threads

// Streaming choices for the value rows (read once) and for H / dV (written
// once), set by measurement on MI355X: non-temporal accesses gave +12% on
// the forward and +9% on the backward at d = 2048, S = 64.
constexpr bool kNtLoad = true;
constexpr bool kNtStore = true;

// Sources whose value rows one lane has in flight in the forward mix.
template <int NCH> struct MixUnroll { static constexpr int value = NCH >= 8 ? 1 : 8 / NCH; };
// Sources loaded ahead in the backward stream (divides 8, the number of
// sources per batched reduction of the dots dH . o_i).
template <int NCH> struct BwdInflight { static constexpr int value = NCH >= 8 ? 1 : NCH >= 2 ? 2 : 4; };
// Tokens per wave in the backward of projected / sliced keys, by column
// chunks per lane: two for rows of 4+ chunks (d >= 2048 bf16), else one
// (measured on MI355X at d = 1024 and 2048).
constexpr int bwd_tokens_per_wave(int nch) { return nch >= 4 ? 2 : 1; }

// ---------------------------------------------------------------------------
// Scores and softmax (Eqs. lr_key_norm and lr_attnres_weight)
// ---------------------------------------------------------------------------

// Lane-per-source scores of token n: rho_i = sqrt(mean_j k_ij^2 + eps),
// s_i = q . k_i / rho_i.  Key element j of source i is
// keys[(i*N + n)*krow + koff + j]  (projected: keys = K, krow = r, koff = 0;
// sliced: keys = V, krow = d, koff = d - r).  Each lane writes only the
// entries of its own sources.
template <typename T, int VEC>
__device__ void lr_scores(const T *__restrict__ keys, const float *__restrict__ q, int S,
                          int N, int r, int krow, int koff, float eps, int n, int lane,
                          float *s_out, float *rho_out)
{
    const bool kvec = VEC > 1 && r % VEC == 0 && krow % VEC == 0 && koff % VEC == 0;
    for (int i = lane; i < S; i += kWaveSize) {
        const T *kp = keys + ((size_t)i * N + n) * krow + koff;
        float ss = 0.0f, dot = 0.0f;
        if (kvec) {
            for (int j = 0; j < r; j += VEC) {
                float x[VEC];
                widen(load_raw<T, VEC>(kp + j), x);
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    ss = fmaf(x[e], x[e], ss);
                    dot = fmaf(q[j + e], x[e], dot);
                }
            }
        } else {
            for (int j = 0; j < r; ++j) {
                const float x = load_elem(kp + j);
                ss = fmaf(x, x, ss);
                dot = fmaf(q[j], x, dot);
            }
        }
        const float rho = sqrtf(ss / (float)r + eps);
        s_out[i] = dot / rho;
        if (rho_out)
            rho_out[i] = rho;
    }
}

// alpha_i = exp(s_i - max) / sum_l exp(s_l - max) over the S sources.
// s and alpha may alias.  Ends with the wave's LDS writes visible.
__device__ void depth_softmax(const float *s, float *alpha, int S, int lane)
{
    float m = -INFINITY;
    for (int i = lane; i < S; i += kWaveSize)
        m = fmaxf(m, s[i]);
    m = wave_max(m);
    float z = 0.0f;
    for (int i = lane; i < S; i += kWaveSize) {
        const float e = expf(s[i] - m);
        alpha[i] = e;
        z += e;
    }
    z = wave_sum(z);
    const float inv = 1.0f / z;
    for (int i = lane; i < S; i += kWaveSize)
        alpha[i] *= inv;
    wave_lds_sync();
}

// ---------------------------------------------------------------------------
// The value stream (Eq. lr_attnres_output): h = sum_i alpha_i o_i
// ---------------------------------------------------------------------------

// vbase points at column (col0 + lane*VEC) of source 0's row of the token;
// chunk c of source i is at vbase + i*plane + c*64*VEC.
template <typename T, int VEC, int NCH, bool FULLCOLS>
__device__ __forceinline__ void mix_rows(const T *__restrict__ vbase, size_t plane, int S,
                                         const float *alpha, const bool (&ok)[NCH],
                                         float (&acc)[NCH][VEC])
{
    typedef typename Raw<T, VEC>::type raw_t;
    constexpr int U = MixUnroll<NCH>::value;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] = 0.0f;
    int i = 0;
    for (; i + U <= S; i += U) {
        raw_t raw[U][NCH];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int c = 0; c < NCH; ++c)
                if (FULLCOLS || ok[c])
                    raw[u][c] = load_stream<T, VEC, kNtLoad>(vbase + (size_t)(i + u) * plane +
                                                             c * kWaveSize * VEC);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float a = alpha[i + u];
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULLCOLS || ok[c]) {
                    float x[VEC];
                    widen(raw[u][c], x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        acc[c][e] = fmaf(a, x[e], acc[c][e]);
                }
            }
        }
    }
    for (; i < S; ++i) {
        const float a = alpha[i];
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (FULLCOLS || ok[c]) {
                float x[VEC];
                widen(load_stream<T, VEC, kNtLoad>(vbase + (size_t)i * plane +
                                                   c * kWaveSize * VEC), x);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    acc[c][e] = fmaf(a, x[e], acc[c][e]);
            }
        }
    }
}

template <typename T, int VEC, int NCH, bool FULLCOLS>
__device__ __forceinline__ void store_row(T *__restrict__ base, const bool (&ok)[NCH],
                                          const float (&acc)[NCH][VEC])
{
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        if (FULLCOLS || ok[c])
            store_stream<T, VEC, kNtStore>(base + c * kWaveSize * VEC,
                                           Narrow<T, VEC>::run(acc[c]));
}

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
template <typename T, int VEC, int NCH, bool FULLCOLS, int KV>
__global__ void __launch_bounds__(kBlock)
route_bwd_lr(const T *__restrict__ V, const T *__restrict__ keys, const float *__restrict__ q,
             const T *__restrict__ dH, T *__restrict__ dV, T *__restrict__ dK,
             float *__restrict__ partial, int S, int N, int d, int r, int krow, int koff,
             int sliced, int tail_start, float eps, int s_pad, int r_pad, int tpw, int lps)
{
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
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

    for (int t = 0; t < tpw; ++t) {
        const int n = (blockIdx.x * tpw + t) * kWaves + wave;
        if (n >= N)
            break;  // wave-uniform; the workgroup barrier below is outside the loop
        lr_scores<T, VEC>(keys, q, S, N, r, krow, koff, eps, n, lane, s, rho);
        depth_softmax(s, alpha, S, lane);

        typedef typename Raw<T, VEC>::type raw_t;
        float dh[NCH][VEC];
        const T *dhrow = dH + (size_t)n * d + col;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (FULLCOLS || ok[c]) {
                widen(load_raw<T, VEC>(dhrow + c * kWaveSize * VEC), dh[c]);
            } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    dh[c][e] = 0.0f;
            }
        }
        const T *vbase = V + (size_t)n * d + col;
        T *dvbase = dV + (size_t)n * d + col;
        constexpr int L = BwdInflight<NCH>::value;
        for (int i0 = 0; i0 < S; i0 += 8) {
            float part[8];
#pragma unroll
            for (int h = 0; h < 8; h += L) {
                raw_t raw[L][NCH];
#pragma unroll
                for (int u = 0; u < L; ++u)
                    if (i0 + h + u < S)
#pragma unroll
                        for (int c = 0; c < NCH; ++c)
                            if (FULLCOLS || ok[c])
                                raw[u][c] = load_stream<T, VEC, kNtLoad>(
                                    vbase + (size_t)(i0 + h + u) * plane + c * kWaveSize * VEC);
#pragma unroll
                for (int u = 0; u < L; ++u) {
                    float p = 0.0f;
                    const int i = i0 + h + u;
                    if (i < S) {
                        const float a = alpha[i];
#pragma unroll
                        for (int c = 0; c < NCH; ++c) {
                            if (FULLCOLS || ok[c]) {
                                float x[VEC], y[VEC];
                                widen(raw[u][c], x);
#pragma unroll
                                for (int e = 0; e < VEC; ++e) {
                                    p = fmaf(dh[c][e], x[e], p);
                                    y[e] = a * dh[c][e];
                                }
                                if (wr[c])
                                    store_stream<T, VEC, kNtStore>(
                                        dvbase + (size_t)i * plane + c * kWaveSize * VEC,
                                        Narrow<T, VEC>::run(y));
                            }
                        }
                    }
                    part[h + u] = p;
                }
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
        gb = wave_sum(gb);
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
                widen(load_raw<T, KV>(dH + (size_t)n * d + c0), dhk);
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
                float x[KV], y[KV];
                if (!sliced) {
                    widen(load_raw<T, KV>(keys + row * krow + c0), x);
#pragma unroll
                    for (int e = 0; e < KV; ++e) {
                        const float kb = x[e] * ri;
                        y[e] = fmaf(cq, qk[k][e], -ck * kb);
                        dq_acc[k][e] = fmaf(dsi, kb, dq_acc[k][e]);
                    }
                    store_raw<T, KV>(dK + row * r + c0, Narrow<T, KV>::run(y));
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
                    store_raw<T, KV>(dV + row * d + c0, Narrow<T, KV>::run(y));
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
        partial[(size_t)blockIdx.x * r + j] = sum;
    }
}

// Full-rank AttnRes backward: pass 1 reads the rows once for sum(o^2), q.o
// and dH.o (one batched reduction per 4 sources); pass 2 re-reads them to
// write dV_i = alpha_i dH + (ds_i/rho_i)(q - o_i s_i/(rho_i d)) and to
// accumulate dq = sum ds_i o_i / rho_i per lane column.
template <typename T, int VEC, int NCH, bool FULLCOLS>
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

    for (int t = 0; t < tpw; ++t) {
        const int n = (blockIdx.x * tpw + t) * kWaves + wave;
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
        partial[(size_t)blockIdx.x * d + j] = stage[j];
}

// dq[j] = sum_b partial[b][j] in a fixed order: one workgroup per column;
// thread t sums rows t, t+256, ... in order, then a fixed pairwise tree over
// the 256 thread sums.  Writes zeros when nblocks = 0.
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
        dq[j] = red[0];
}

// ---------------------------------------------------------------------------
// Host side: plan selection and launches
// ---------------------------------------------------------------------------

namespace {

constexpr int kMaxSourcesFwd = 1024;
constexpr int kMaxSourcesBwd = 512;
constexpr int kMaxRankBwd = 256;

int round_up(int x, int m) { return (x + m - 1) / m * m; }

struct Plan {
    int vec = 1;          // elements per lane access
    int nch = 1;          // column chunks per lane
    bool fullcols = false;
    int ysplit = 1;       // column blocks (forward, projected/sliced only)
    int tpw = 1;          // tokens per wave (backward)
    int nblocks = 0;      // workgroups along x
    int s_pad = 4;
    int r_pad = 4;
    size_t lds = 0;
};

bool make_plan(const Problem &p, bool bwd, Plan *pl, std::string *why)
{
    const int vmax = p.dtype == LRAR_DTYPE_BF16 ? 8 : 4;
    pl->vec = p.d % vmax == 0 ? vmax : 1;
    const int width = kWaveSize * pl->vec;
    const int64_t need = (p.d + width - 1) / width;
    static const int vec_list[] = {1, 2, 4, 8};
    static const int sc_list[] = {1, 2, 4, 8, 16};
    const int *list = pl->vec > 1 ? vec_list : sc_list;
    const int nlist = pl->vec > 1 ? 4 : 5;
    const int maxch = list[nlist - 1];
    if (p.N > (1 << 30)) {
        *why = "N exceeds 2^30 tokens";
        return false;
    }
    if (p.S > (bwd ? kMaxSourcesBwd : kMaxSourcesFwd)) {
        *why = bwd ? "backward supports at most 512 sources" : "forward supports at most 1024 sources";
        return false;
    }
    if (bwd && p.mode != LRAR_MODE_FULL && p.r > kMaxRankBwd) {
        *why = "backward with projected or sliced keys supports r <= 256";
        return false;
    }
    if (need > maxch) {
        if (bwd || p.mode == LRAR_MODE_FULL) {
            *why = "row width d too large for the backward / full-rank kernels";
            return false;
        }
        pl->nch = maxch;
        pl->ysplit = (int)((need + maxch - 1) / maxch);
    } else {
        for (int k = 0; k < nlist; ++k)
            if (list[k] >= need) {
                pl->nch = list[k];
                break;
            }
    }
    pl->fullcols = pl->vec > 1 && p.d % ((int64_t)width * pl->nch) == 0;
    pl->s_pad = round_up((int)p.S, 4);
    pl->r_pad = round_up((int)p.r, 4);
    if (!bwd) {
        pl->nblocks = (int)((p.N + kWaves - 1) / kWaves);
        // The low-rank forward keeps the weights in LDS; the full-rank one
        // holds its online-softmax state in registers.
        pl->lds = p.mode == LRAR_MODE_FULL ? 0 : (size_t)kWaves * pl->s_pad * sizeof(float);
    } else {
        pl->tpw = p.mode == LRAR_MODE_FULL ? 4 : bwd_tokens_per_wave(pl->nch);
        const int64_t per_block = (int64_t)kWaves * pl->tpw;
        pl->nblocks = (int)((p.N + per_block - 1) / per_block);
        pl->lds = (size_t)kWaves * 4 * pl->s_pad * sizeof(float);
        pl->lds += p.mode == LRAR_MODE_FULL ? (size_t)round_up((int)p.d, 4) * sizeof(float)
                                            : (size_t)kWaves * pl->r_pad * sizeof(float);
    }
    return true;
}

// Calls f(std::integral_constant<int, NCH>, std::integral_constant<bool, FULLCOLS>).
template <int VEC, typename F>
hipError_t dispatch_chunks(const Plan &pl, F &&f)
{
    typedef std::true_type Y;
    typedef std::false_type Nf;
    if constexpr (VEC > 1) {
        switch (pl.nch) {
        case 1: return pl.fullcols ? f(std::integral_constant<int, 1>{}, Y{}) : f(std::integral_constant<int, 1>{}, Nf{});
        case 2: return pl.fullcols ? f(std::integral_constant<int, 2>{}, Y{}) : f(std::integral_constant<int, 2>{}, Nf{});
        case 4: return pl.fullcols ? f(std::integral_constant<int, 4>{}, Y{}) : f(std::integral_constant<int, 4>{}, Nf{});
        case 8: return pl.fullcols ? f(std::integral_constant<int, 8>{}, Y{}) : f(std::integral_constant<int, 8>{}, Nf{});
        }
    } else {
        switch (pl.nch) {
        case 1: return f(std::integral_constant<int, 1>{}, Nf{});
        case 2: return f(std::integral_constant<int, 2>{}, Nf{});
        case 4: return f(std::integral_constant<int, 4>{}, Nf{});
        case 8: return f(std::integral_constant<int, 8>{}, Nf{});
        case 16: return f(std::integral_constant<int, 16>{}, Nf{});
        }
    }
    return hipErrorInvalidValue;
}

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

template <typename T, int VEC>
hipError_t launch_bwd_t(const Problem &p, const Plan &pl, const void *dH, void *dV, void *dK,
                        float *partial, hipStream_t st)
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
        if (p.mode == LRAR_MODE_FULL) {
            hipLaunchKernelGGL((route_bwd_full<T, VEC, NCH, FC>), dim3(pl.nblocks), dim3(kBlock),
                               pl.lds, st, V, p.q, static_cast<const T *>(dH),
                               static_cast<T *>(dV), partial, (int)p.S, (int)p.N, (int)p.d,
                               p.eps, pl.s_pad, pl.tpw);
            return hipGetLastError();
        }
        auto launch = [&](auto kvc) {
            constexpr int KV = decltype(kvc)::value;
            hipLaunchKernelGGL((route_bwd_lr<T, VEC, NCH, FC, KV>), dim3(pl.nblocks),
                               dim3(kBlock), pl.lds, st, V, keys, p.q,
                               static_cast<const T *>(dH), static_cast<T *>(dV),
                               static_cast<T *>(dK), partial, (int)p.S, (int)p.N, (int)p.d,
                               (int)p.r, krow, koff, p.mode == LRAR_MODE_SLICED ? 1 : 0,
                               tail_start, p.eps, pl.s_pad, pl.r_pad, pl.tpw, kp.lps);
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

int hip_status(hipError_t e, const char *what, std::string *err)
{
    if (e == hipSuccess)
        return LRAR_OK;
    *err = std::string(what) + ": " + hipGetErrorString(e);
    return LRAR_EHIP;
}

}  // namespace

int check_supported(const Problem &p, bool bwd, std::string *why)
{
    Plan pl;
    return make_plan(p, bwd, &pl, why) ? LRAR_OK : LRAR_EUNSUPPORTED;
}

size_t bwd_workspace_bytes(const Problem &p)
{
    Plan pl;
    std::string why;
    if (!make_plan(p, true, &pl, &why))
        return 0;
    const int64_t ncols = p.mode == LRAR_MODE_FULL ? p.d : p.r;
    return (size_t)pl.nblocks * (size_t)ncols * sizeof(float);
}

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

int launch_bwd(const Problem &p, const void *dH, void *dV, void *dK, float *dq, void *ws,
               hipStream_t st, std::string *err)
{
    Plan pl;
    if (!make_plan(p, true, &pl, err))
        return LRAR_EUNSUPPORTED;
    float *partial = static_cast<float *>(ws);
    hipError_t e = hipSuccess;
    if (p.N > 0) {
        if (p.dtype == LRAR_DTYPE_BF16)
            e = pl.vec > 1 ? launch_bwd_t<uint16_t, 8>(p, pl, dH, dV, dK, partial, st)
                           : launch_bwd_t<uint16_t, 1>(p, pl, dH, dV, dK, partial, st);
        else
            e = pl.vec > 1 ? launch_bwd_t<float, 4>(p, pl, dH, dV, dK, partial, st)
                           : launch_bwd_t<float, 1>(p, pl, dH, dV, dK, partial, st);
        if (e != hipSuccess)
            return hip_status(e, "route_bwd launch", err);
    }
    const int ncols = (int)(p.mode == LRAR_MODE_FULL ? p.d : p.r);
    const int nb = p.N > 0 ? pl.nblocks : 0;
    hipLaunchKernelGGL(dq_reduce, dim3(ncols), dim3(256), 0, st, partial, dq, nb,
                       ncols);
    return hip_status(hipGetLastError(), "dq_reduce launch", err);
}

}  // namespace lrar
