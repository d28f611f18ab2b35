#pragma once
// Shared pieces of the gfx950 LR-AttnRes depth-routing kernels (arXiv
// 2607.09694, Sec. 3): tiling constants, the score / softmax / value-stream
// device building blocks, and the launch plan shared by the host launchers.
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
// s_waitcnt immediate (gfx9 encoding) that waits for this wave's LDS
// accesses only (lgkmcnt 0; vmcnt and expcnt at their maxima).
constexpr int kWaitLdsOnly = 0x000F | (0x7 << 4) | (0x0 << 8) | (0x3 << 14);

// Workgroup barrier that orders LDS only: this wave's LDS accesses complete,
// then s_barrier.  Unlike __syncthreads it does not wait for outstanding
// global loads, so loads issued ahead stay in flight across it.  The
// kernels that use it communicate between waves through LDS alone.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(kWaitLdsOnly);
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The workgroup a launched one stands for, so that each of the 8 XCDs of
// the chip holds one contiguous range of the grid (row-major linear index
// x + y * gridDim.x).  The hardware deals workgroups to the XCDs round-robin
// (linear index mod 8); remapped, the rows an XCD reads at one time come
// from one token range of each source plane.  Streams over the planes ran
// about 10% faster this way on MI355X (reads of 49 planes at d = 1024:
// 6.2 -> 6.9 TB/s).  A bijection of the grid for any size.
constexpr int kXcds = 8;
struct BlockXY {
    int x, y;
};
__device__ __forceinline__ BlockXY xcd_block()
{
    const int nx = (int)gridDim.x, total = nx * (int)gridDim.y;
    const int b = (int)blockIdx.x + (int)blockIdx.y * nx;
    const int xcd = b % kXcds, i = b / kXcds;
    const int full = total / kXcds, rem = total % kXcds;
    const int m = xcd * full + min(xcd, rem) + i;
    return BlockXY{m % nx, m / nx};
}

template <int NCH> struct MixUnroll { static constexpr int value = NCH >= 8 ? 1 : 8 / NCH; };
// Sources loaded per step of the backward stream (divides 8, the number of
// sources per batched reduction of the dots dH . o_i).  At d = 2048 one
// source per step (4 KB read, 4 KB written per wave) measured level with or
// ahead of two on MI355X; both sit at the box's read + write copy rate.
#ifndef LRAR_BWD_INFLIGHT_WIDE
#define LRAR_BWD_INFLIGHT_WIDE 1  // rows of 4 chunks per lane (d = 2048 bf16)
#endif
template <int NCH> struct BwdInflight {
    static constexpr int value = NCH >= 8 ? 1 : NCH == 4 ? LRAR_BWD_INFLIGHT_WIDE : NCH >= 2 ? 2 : 4;
};
// Cache policy of the backward's value-row loads and gradient-row stores.
#ifndef LRAR_BWD_NT_LOAD
#define LRAR_BWD_NT_LOAD 1
#endif
#ifndef LRAR_BWD_NT_STORE
#define LRAR_BWD_NT_STORE 1
#endif
constexpr bool kBwdNtLoad = LRAR_BWD_NT_LOAD != 0;
constexpr bool kBwdNtStore = LRAR_BWD_NT_STORE != 0;
// Tokens per wave in the backward of projected / sliced keys, by column
// chunks per lane: two for rows of 4+ chunks (d >= 2048 bf16), else one
// (measured on MI355X at d = 1024 and 2048).
constexpr int bwd_tokens_per_wave(int nch) { return nch >= 4 ? 2 : 1; }

// Tokens per wave (TW) and sources per load batch (SB) of the forward of
// projected / sliced keys.  A wave owns TW consecutive tokens, whose rows are
// adjacent in every source plane, and each round trip loads SB sources
// across them: SB plane visits of TW * 2d contiguous bytes.  Measured on
// MI355X (49 planes, d = 1024, cold), the shape of that batch sets the read
// rate: 2 tokens x 1 source ran at 6.5 TB/s, 1 token x 4 sources at 6.1,
// and keeping a second batch in flight (two register buffers) was slower
// in every shape tried.
#ifndef LRAR_FWD_TW_NARROW
#define LRAR_FWD_TW_NARROW 2  // rows of at most 2 chunks per lane (d <= 1024 bf16)
#endif
#ifndef LRAR_FWD_SB_NARROW
#define LRAR_FWD_SB_NARROW 1
#endif
#ifndef LRAR_FWD_TW_WIDE
#define LRAR_FWD_TW_WIDE 2    // rows of 4 chunks (d <= 2048 bf16)
#endif
#ifndef LRAR_FWD_SB_WIDE
#define LRAR_FWD_SB_WIDE 1
#endif
constexpr int fwd_tokens_per_wave(int nch)
{
    return nch <= 2 ? LRAR_FWD_TW_NARROW : nch == 4 ? LRAR_FWD_TW_WIDE : 1;
}
constexpr int fwd_sources_per_batch(int nch)
{
    return nch <= 2 ? LRAR_FWD_SB_NARROW : nch == 4 ? LRAR_FWD_SB_WIDE : 1;
}
#ifndef LRAR_FWD_LPR_NARROW
#define LRAR_FWD_LPR_NARROW 2
#endif
#ifndef LRAR_FWD_LPR_WIDE
#define LRAR_FWD_LPR_WIDE 2
#endif
constexpr int fwd_loads_per_trip(int nch)
{
    return nch <= 2 ? LRAR_FWD_LPR_NARROW : nch == 4 ? LRAR_FWD_LPR_WIDE : 2;
}

// ---------------------------------------------------------------------------
// Scores and softmax (Eqs. lr_key_norm and lr_attnres_weight)
// ---------------------------------------------------------------------------

// Scores of token n: rho_i = sqrt(mean_j k_ij^2 + eps), s_i = q . k_i / rho_i.
// Key element j of source i is keys[(i*N + n)*krow + koff + j] (projected:
// keys = K, krow = r, koff = 0; sliced: keys = V, krow = d, koff = d - r).
// The key of one source is nkv vectors of KV elements; a group of lps lanes
// (the power of two >= nkv, at most 64) reads one source's key, each lane its
// vectors, and the group sums its partial dot products with lps-lane
// butterflies, so 64 / lps sources are scored per step.  The group's first
// lane writes s_out[i] (and rho_out[i]).
// DPP: the lane-group butterflies with DPP moves (butterfly_sum2; same
// bits).  Measured on MI355X: faster in the backward over fp32 block slots
// (1-2% on the block reverse passes), slower in the bf16 forward and the
// fp32 block forward, which keep the LDS lane permutes.
template <typename T, int KV, bool DPP = false>
__device__ inline void lr_scores_kv(const T *__restrict__ keys, const float *__restrict__ q,
                                    int S, int N, int r, int krow, int koff, float eps, int n,
                                    int lane, float *s_out, float *rho_out)
{
    const int nkv = r / KV;
    int lps = 1;
    while (lps < nkv && lps < kWaveSize)
        lps <<= 1;
    const int spi = kWaveSize / lps;
    const int isub = lane / lps, v = lane % lps;
    if (nkv <= lps) {
        // At most one key vector per lane and source: the loads of KP
        // groups of sources go out together (sources past S re-read source
        // S-1 and lanes past the key re-read its last vector; neither
        // counts), then the scores of the KP groups are formed.
        constexpr int KP = 4;
        typedef typename Raw<T, KV>::type raw_t;
        const bool vok = v < nkv;
        const int vv = min(v, nkv - 1);
        float qv[KV];
#pragma unroll
        for (int e = 0; e < KV; ++e)
            qv[e] = vok ? q[vv * KV + e] : 0.0f;
        for (int i0 = 0; i0 < S; i0 += KP * spi) {
            raw_t kr[KP];
#pragma unroll
            for (int p = 0; p < KP; ++p) {
                const int i = min(i0 + p * spi + isub, S - 1);
                kr[p] = load_raw<T, KV>(keys + ((size_t)i * N + n) * krow + koff + vv * KV);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int p = 0; p < KP; ++p) {
                float x[KV];
                widen(kr[p], x);
                float ss = 0.0f, dot = 0.0f;
#pragma unroll
                for (int e = 0; e < KV; ++e) {
                    ss = fmaf(x[e], x[e], ss);
                    dot = fmaf(qv[e], x[e], dot);
                }
                if (!vok)
                    ss = dot = 0.0f;
                butterfly_sum2<DPP>(ss, dot, lps);
                const int i = i0 + p * spi + isub;
                if (v == 0 && i < S) {
                    const float rho = sqrtf(ss / (float)r + eps);
                    s_out[i] = dot / rho;
                    if (rho_out)
                        rho_out[i] = rho;
                }
            }
        }
        return;
    }
    for (int i0 = 0; i0 < S; i0 += spi) {
        const int i = i0 + isub;
        float ss = 0.0f, dot = 0.0f;
        if (i < S) {
            const T *kp = keys + ((size_t)i * N + n) * krow + koff;
            for (int vv = v; vv < nkv; vv += lps) {
                float x[KV];
                widen(load_raw<T, KV>(kp + vv * KV), x);
#pragma unroll
                for (int e = 0; e < KV; ++e) {
                    ss = fmaf(x[e], x[e], ss);
                    dot = fmaf(q[vv * KV + e], x[e], dot);
                }
            }
        }
        butterfly_sum2<DPP>(ss, dot, lps);
        if (v == 0 && i < S) {
            const float rho = sqrtf(ss / (float)r + eps);
            s_out[i] = dot / rho;
            if (rho_out)
                rho_out[i] = rho;
        }
    }
}

// The scores with 16-byte key vectors when the key rows allow them, else
// element by element.  Ends with the wave's LDS writes visible.
template <typename T, int VEC, bool DPP = false>
__device__ inline void lr_scores(const T *__restrict__ keys, const float *__restrict__ q, int S,
                                 int N, int r, int krow, int koff, float eps, int n, int lane,
                                 float *s_out, float *rho_out)
{
    if (VEC > 1 && r % VEC == 0 && krow % VEC == 0 && koff % VEC == 0)
        lr_scores_kv<T, VEC, DPP>(keys, q, S, N, r, krow, koff, eps, n, lane, s_out, rho_out);
    else
        lr_scores_kv<T, 1, DPP>(keys, q, S, N, r, krow, koff, eps, n, lane, s_out, rho_out);
    wave_lds_sync();
}

// Scores of the TW consecutive tokens n0 .. n0+TW-1 into s_out[t * s_pad + i]
// (tokens at or past N are read as token N-1 and not written).  With at most
// one key vector per lane and source, the key loads of all TW tokens and KP
// groups of sources go out together; otherwise token by token.
template <typename T, int KV, int TW>
__device__ inline void lr_scores_tokens_kv(const T *__restrict__ keys, const float *__restrict__ q,
                                           int S, int N, int r, int krow, int koff, float eps,
                                           int n0, int lane, float *s_out, int s_pad)
{
    const int nkv = r / KV;
    int lps = 1;
    while (lps < nkv && lps < kWaveSize)
        lps <<= 1;
    if (nkv > lps) {
        for (int t = 0; t < TW; ++t)
            if (n0 + t < N)
                lr_scores_kv<T, KV>(keys, q, S, N, r, krow, koff, eps, n0 + t, lane,
                                    s_out + t * s_pad, nullptr);
        return;
    }
    constexpr int KP = TW >= 4 ? 1 : TW == 2 ? 2 : 4;
    typedef typename Raw<T, KV>::type raw_t;
    const int spi = kWaveSize / lps;
    const int isub = lane / lps, v = lane % lps;
    const bool vok = v < nkv;
    const int vv = min(v, nkv - 1);
    float qv[KV];
#pragma unroll
    for (int e = 0; e < KV; ++e)
        qv[e] = vok ? q[vv * KV + e] : 0.0f;
    for (int i0 = 0; i0 < S; i0 += KP * spi) {
        raw_t kr[TW][KP];
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int n = min(n0 + t, N - 1);
#pragma unroll
            for (int p = 0; p < KP; ++p) {
                const int i = min(i0 + p * spi + isub, S - 1);
                kr[t][p] = load_raw<T, KV>(keys + ((size_t)i * N + n) * krow + koff + vv * KV);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < TW; ++t) {
#pragma unroll
            for (int p = 0; p < KP; ++p) {
                float x[KV];
                widen(kr[t][p], x);
                float ss = 0.0f, dot = 0.0f;
#pragma unroll
                for (int e = 0; e < KV; ++e) {
                    ss = fmaf(x[e], x[e], ss);
                    dot = fmaf(qv[e], x[e], dot);
                }
                if (!vok)
                    ss = dot = 0.0f;
                butterfly_sum2<false>(ss, dot, lps);
                const int i = i0 + p * spi + isub;
                if (v == 0 && i < S && n0 + t < N)
                    s_out[t * s_pad + i] = dot / sqrtf(ss / (float)r + eps);
            }
        }
    }
}

template <typename T, int VEC, int TW>
__device__ inline void lr_scores_tokens(const T *__restrict__ keys, const float *__restrict__ q,
                                        int S, int N, int r, int krow, int koff, float eps,
                                        int n0, int lane, float *s_out, int s_pad)
{
    if (VEC > 1 && r % VEC == 0 && krow % VEC == 0 && koff % VEC == 0)
        lr_scores_tokens_kv<T, VEC, TW>(keys, q, S, N, r, krow, koff, eps, n0, lane, s_out,
                                        s_pad);
    else
        lr_scores_tokens_kv<T, 1, TW>(keys, q, S, N, r, krow, koff, eps, n0, lane, s_out, s_pad);
    wave_lds_sync();
}

// alpha_i = exp(s_i - max) / sum_l exp(s_l - max) over the S sources.
// s and alpha may alias.  Ends with the wave's LDS writes visible.  DPP: the
// wave reductions with DPP moves (wave_sum_t), used over fp32 block slots.
template <bool DPP = false>
__device__ inline void depth_softmax(const float *s, float *alpha, int S, int lane)
{
    float m = -INFINITY;
    for (int i = lane; i < S; i += kWaveSize)
        m = fmaxf(m, s[i]);
    m = wave_max_t<DPP>(m);
    float z = 0.0f;
    for (int i = lane; i < S; i += kWaveSize) {
        const float e = expf(s[i] - m);
        alpha[i] = e;
        z += e;
    }
    z = wave_sum_t<DPP>(z);
    const float inv = 1.0f / z;
    for (int i = lane; i < S; i += kWaveSize)
        alpha[i] *= inv;
    wave_lds_sync();
}

// ---------------------------------------------------------------------------
// The value stream (Eq. lr_attnres_output): h = sum_i alpha_i o_i
// ---------------------------------------------------------------------------

// vbase points at column (col0 + lane*VEC) of source 0's row of the token;
// chunk c of source i is at vbase + i*plane + c*64*VEC.  acc starts at zero,
// or (CONTINUE) goes on from the sum it holds, in source order.
template <typename T, int VEC, int NCH, bool FULLCOLS, bool CONTINUE = false>
__device__ __forceinline__ void mix_rows(const T *__restrict__ vbase, size_t plane, int S,
                                         const float *alpha, const bool (&ok)[NCH],
                                         float (&acc)[NCH][VEC])
{
    typedef typename Raw<T, VEC>::type raw_t;
    constexpr int U = MixUnroll<NCH>::value;
    if constexpr (!CONTINUE) {
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                acc[c][e] = 0.0f;
    }
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
        // Keep the batch's loads together ahead of their uses: without this
        // the scheduler sinks each load next to its first use, leaving one
        // source's row in flight at a time.
        __builtin_amdgcn_sched_barrier(0);
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

// The same stream with two batches of U sources in registers: the loads of
// batch b + 1 are issued before batch b is multiplied, so a wave keeps
// between U and 2U rows in flight instead of draining to none between
// batches.  Batch 0 is loaded by the caller into ra (mix_batch_load), which
// lets it go out before the scores are known.  Loads past the last source
// re-read source S-1 (the same lines, in flight together; no HBM traffic of
// their own) and are not accumulated: with every load unconditional, the
// compiler's wait counts leave the newer batch in flight while the older
// one is used.  Sums in source order, like mix_rows (bit-identical).
template <typename T, int VEC, int NCH, bool FULLCOLS, int U>
__device__ __forceinline__ void mix_batch_load(typename Raw<T, VEC>::type (&r)[U][NCH],
                                               const T *__restrict__ vbase, size_t plane, int i,
                                               int S, const bool (&ok)[NCH])
{
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int src = min(i + u, S - 1);
#pragma unroll
        for (int c = 0; c < NCH; ++c)
            if (FULLCOLS || ok[c])
                r[u][c] = load_stream<T, VEC, kNtLoad>(vbase + (size_t)src * plane +
                                                       c * kWaveSize * VEC);
    }
}

template <typename T, int VEC, int NCH, bool FULLCOLS, int U>
__device__ __forceinline__ void mix_batch_fma(const typename Raw<T, VEC>::type (&r)[U][NCH],
                                              const float *alpha, int i, int S,
                                              const bool (&ok)[NCH], float (&acc)[NCH][VEC])
{
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (i + u < S) {
            const float a = alpha[i + u];
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                if (FULLCOLS || ok[c]) {
                    float x[VEC];
                    widen(r[u][c], x);
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        acc[c][e] = fmaf(a, x[e], acc[c][e]);
                }
            }
        }
    }
}

template <typename T, int VEC, int NCH, bool FULLCOLS, int U>
__device__ __forceinline__ void mix_rows_pipelined(typename Raw<T, VEC>::type (&ra)[U][NCH],
                                                   const T *__restrict__ vbase, size_t plane,
                                                   int S, const float *alpha,
                                                   const bool (&ok)[NCH], float (&acc)[NCH][VEC])
{
    typename Raw<T, VEC>::type rb[U][NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            acc[c][e] = 0.0f;
    // ra holds batch 0 (sources 0 .. U-1) on entry; nb batches in all.
    const int nb = (S + U - 1) / U;
    int b = 0;
    for (; b + 2 < nb; b += 2) {
        mix_batch_load<T, VEC, NCH, FULLCOLS, U>(rb, vbase, plane, (b + 1) * U, S, ok);
        __builtin_amdgcn_sched_barrier(0);
        mix_batch_fma<T, VEC, NCH, FULLCOLS, U>(ra, alpha, b * U, S, ok, acc);
        mix_batch_load<T, VEC, NCH, FULLCOLS, U>(ra, vbase, plane, (b + 2) * U, S, ok);
        __builtin_amdgcn_sched_barrier(0);
        mix_batch_fma<T, VEC, NCH, FULLCOLS, U>(rb, alpha, (b + 1) * U, S, ok, acc);
    }
    if (b + 1 < nb) {
        mix_batch_load<T, VEC, NCH, FULLCOLS, U>(rb, vbase, plane, (b + 1) * U, S, ok);
        __builtin_amdgcn_sched_barrier(0);
        mix_batch_fma<T, VEC, NCH, FULLCOLS, U>(ra, alpha, b * U, S, ok, acc);
        mix_batch_fma<T, VEC, NCH, FULLCOLS, U>(rb, alpha, (b + 1) * U, S, ok, acc);
    } else {
        mix_batch_fma<T, VEC, NCH, FULLCOLS, U>(ra, alpha, b * U, S, ok, acc);
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
// Launch plan (host)
// ---------------------------------------------------------------------------

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
    bool wg_split = false;  // forward: the sources of a token split over a workgroup
};

// Fills *pl for a validated problem, or returns false with the reason.
bool make_plan(const Problem &p, bool bwd, Plan *pl, std::string *why);

// Switches a forward plan to one token per workgroup, its sources split
// over the waves (route_fwd_lr_wg, route_fwd_full_1p<kFullWg>), when the
// tokens are too few to fill the device with one wave each.
void plan_wg_split(const Problem &p, Plan *pl);

// LRAR_OK, or LRAR_EHIP with the HIP error text in *err.
int hip_status(hipError_t e, const char *what, std::string *err);

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

}  // namespace lrar
