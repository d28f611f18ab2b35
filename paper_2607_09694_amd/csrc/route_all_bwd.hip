// Backward of every read site of a pass over one source stack (the gradient
// of the all-sites forward; the paper states no backward).  Site j reads the
// first first+j sources (Sec. 3.1, Eq. full_attnres_source_set) with the
// low-rank keys of Sec. 3.2-3.4.  For the loss L = sum_j sum_n dH_j . h_j,
// per token n, with G[j][i] = dH_j . o_i (the value dots of every site
// against every source):
//     ds[j][i] = alpha[j][i] (G[j][i] - sum_l alpha[j][l] G[j][l]),
//     dV_i     = sum_j alpha[j][i] dH_j                 (+ key path, S-LR),
//     dk_i     = (1 / rho_i) (u_i - kbar_i (kbar_i . u_i) / r),
//                u_i = sum_j ds[j][i] Q_j,
//     dQ_j     = sum_n sum_i ds[j][i] kbar_i.
// (The RMSNorm term kbar_i s_{j,i} / r of each site's key gradient sums to
// kbar_i (kbar_i . u_i) / r, because s_{j,i} = Q_j . kbar_i.)  The stack and
// the upstream gradients are each read once and dV is written once, instead
// of once per site: sum_j (first + j) rows each of V, dV in and dV out.
//
// Per token, on the matrix cores:
//     G  = dH_n [T x d] * O_n^T [d x S]      (v_mfma_f32_16x16x32_bf16, exact
//                                            products of bf16 operands),
//     dV = alpha^T [S x T] * dH_n [T x d]    (alpha as hi + lo bf16, two MFMAs,
//                                            as in the forward),
//     u  = ds^T [S x T] * Q [T x r]          (ds and Q as hi + lo bf16, three
//                                            MFMAs: hi.hi + hi.lo + lo.hi),
//     dQ += (ds / rho) [T x S] * K [S x r]   (ds / rho as hi + lo, the keys
//                                            exact in bf16, two MFMAs).
// Workgroups (4 waves, two per CU) are persistent over a stride of tokens
// and keep their share of dQ in registers; a fixed-order reduction adds the
// per-workgroup partials, so dQ is bitwise reproducible.  Wave w owns
// sources 16 w .. 16 w + 15.  The row is processed in 128-column slabs: the
// workgroup stages the T upstream rows of a slab in LDS (rows padded by one
// 16-byte chunk, conflict-free in both read patterns below), each wave
// loads its 16 source rows of the slab into registers, then
//   - G: A = dH rows from LDS (lane: one site, 8 columns), B = the source
//     rows (lane: one source, the same 8 columns);
//   - dV: A = alpha^T (lane: one source, 8 sites), B = dH read from LDS as 8
//     site rows x 8 consecutive columns per lane and transposed in registers,
//     so that the p-th MFMA's column index stands for column c0 + p; the
//     result is 8 consecutive columns of 4 sources per lane, stored as
//     16-byte rows.
// The next slab is loaded while the current one is multiplied; the other
// workgroup on the CU covers the per-token phases (scores, key gradients).
// With sliced keys the key gradient lands in the last r columns of dV, which
// needs the whole of G first: those columns' value gradients wait in LDS in
// fp32 (where the weights were) and are rounded once the key gradient has
// been added.  Workgroup barriers here order LDS only (lds_barrier), so
// loads issued ahead stay in flight across them.
#include "route_all_weights.h"

#include <algorithm>

namespace lrar {

namespace {

constexpr int kAllBwdGrid = 512;                       // persistent workgroups
constexpr int kDhRowBytes = kAllSlab * 2 + 16;         // one slab row of dH, bf16, padded
constexpr int kDhBufBytes = kAllMaxSources * kDhRowBytes;
constexpr int kTailRow = 64;                           // floats per source: key-column octets

struct AllBwdArgs {
    AllArgs f;           // V, keys, Q, sizes (H and neff unused)
    const uint16_t *dH;  // [T][N][d]
    uint16_t *dV;        // [S][N][d]
    uint16_t *dK;        // [S][N][r] (projected keys) or NULL
    float *partial;      // [gridDim.x][T][r]
    bool sliced;         // the key is the last r columns of each value row
};

// LDS byte offset of 16-byte chunk c (0..15) of slab row `row`: rows of 256
// bytes are laid out 272 bytes apart, so both 16 consecutive rows at one
// chunk and one row's 16 chunks fall on distinct banks, and the offsets of
// the rows a lane reads differ by constants (immediate offsets, no per-read
// address arithmetic).
__device__ __forceinline__ int dh_chunk(int row, int c) { return row * kDhRowBytes + 16 * c; }

__device__ __forceinline__ float bf16_at(const uint16_t *p) { return __uint_as_float((unsigned)*p << 16); }

// 8 fp32 values as an MFMA operand pair: hi = RNE(v), lo = RNE(v - hi), so
// that hi + lo carries v to a relative 2^-17.
__device__ __forceinline__ void split_hilo(const float (&v)[8], bf16x8_t &hi, bf16x8_t &lo)
{
    u32x4_t h, l;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const unsigned w = pack_bf16x2(v[2 * k], v[2 * k + 1]);
        h[k] = w;
        l[k] = pack_bf16x2(v[2 * k] - bf16_lo(w), v[2 * k + 1] - bf16_hi(w));
    }
    hi = __builtin_bit_cast(bf16x8_t, h);
    lo = __builtin_bit_cast(bf16x8_t, l);
}

// Keep x opaque to the optimiser for one token: the per-token control flow
// (masks of sites, sources and columns, row offsets) is then formed inside
// the token loop instead of being hoisted out of it and held in registers
// for the workgroup's lifetime.
template <typename T>
__device__ __forceinline__ void per_token(T &x)
{
    asm volatile("" : "+s"(x));
}

// The same for per-lane values: the LDS offsets and masks derived from the
// lane's indices are formed where they are used instead of being
// precomputed once and held (and spilled) for the kernel's lifetime.
__device__ __forceinline__ void per_lane(int &x)
{
    asm volatile("" : "+v"(x));
}

template <int MT, int RT, bool ACC>
__global__ __launch_bounds__(kBlock, 2) void route_all_bwd_bf16(AllBwdArgs b)
{
    constexpr int KG = (MT + 1) / 2;      // groups of 32 sites in the dV contraction
    constexpr int RP = RT <= 2 ? 32 : 64; // key elements covered by the score MFMAs
    constexpr int KK = RP / 32;
    // alpha: the weights, then (sliced keys) the fp32 value gradient of the
    // key columns [16 w + e][c - tail0].  dhbuf: the upstream slabs, then
    // ds / rho [site][source] for dQ.
    __shared__ __align__(16) float alpha[kAllMaxSources * kAlphaRow];
    __shared__ __align__(16) unsigned char dhbuf[2 * kDhBufBytes];
    __shared__ __align__(16) uint16_t keys[kAllMaxSources * kKeyRow];
    __shared__ float rho[kAllMaxSources];
    __shared__ float gpart[kWaves * kAllMaxSources];
    __shared__ float qs[kAllMaxSources * kAllMaxRank];  // Q [T][r]
    static_assert(2 * kDhBufBytes >= kAllMaxSources * kAlphaRow * 4, "ds / rho fits the slabs");

    const int tid0 = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid0 / kWaveSize);
    float *dsr = reinterpret_cast<float *>(dhbuf);
    float *tailbuf = alpha + wave * 16 * kTailRow;  // this wave's 16 sources

    for (int f = tid0; f < b.f.T * b.f.r; f += kBlock)
        qs[f] = b.f.Q[f];

    f32x4_t dq[RT];
#pragma unroll
    for (int ct = 0; ct < RT; ++ct)
        dq[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // The keys of the workgroup's next token are loaded once its current
    // token's slabs are done, so that they arrive during the key-gradient
    // phases instead of holding up the next token's scores.
    u32x4_t kown[4 * KK];
    if (blockIdx.x < b.f.N)
        load_site_keys<RP>(b.f, blockIdx.x, kown);

    for (int64_t n = blockIdx.x; n < b.f.N; n += gridDim.x) {
        int tid = tid0;
        per_lane(tid);
        const int lane = tid % kWaveSize;
        int lc = lane & 15, ks = lane >> 4;
        int src = 16 * wave + lc;  // this lane's source as a G operand
        int hch = tid & 15, hr0 = tid >> 4;
        AllArgs a = b.f;
        per_token(a.S);
        per_token(a.T);
        per_token(a.first);
        per_token(a.r);
        per_token(a.d);
        per_token(a.krow);
        per_token(a.koff);
        per_token(a.N);
        const size_t plane = (size_t)a.N * a.d;
        const int nslab = (a.d + kAllSlab - 1) / kAllSlab;
        const float inv_r = 1.0f / (float)a.r;
        // First column of the key octets (sliced keys; d past the row otherwise).
        const int tail0 = b.sliced ? (a.d - a.r) / 8 * 8 : a.d;

        // Slab loads: thread t brings chunk t mod 16 of dH rows t / 16 + 16 q
        // (q < MT), and lane (lc, ks) the 4 chunks 4 u + ks of its source
        // row.  Lanes past the rows or columns load a valid address (the
        // token's first chunk), so no load sits behind a branch; the
        // consumers (the LDS write of dH, the G operands of V) put zeros in
        // their place, so that no load is waited for early.  The next slab is
        // in flight while the current one is multiplied.  A source row's
        // 128-byte lines are read by two loads (64 bytes of each of 16 rows
        // per load), so those loads go through the caches normally; the
        // upstream rows, read as whole lines, stream.
        u32x4_t hraw[MT], vraw[4];
        // Each lane forms one 64-bit row address per slab; the rows it
        // reads after that are whole planes (16 sites) or 32 columns further
        // on, uniform steps.
        auto load_dh = [&](int s) {
            const int col = s * kAllSlab + 8 * hch;
            const uint16_t *hbase = b.dH + n * a.d;
            const uint16_t *h0 = hbase + (size_t)(unsigned)hr0 * plane + col;
#pragma unroll
            for (int q = 0; q < MT; ++q) {
                const int row = hr0 + 16 * q;
                const bool ok = row < a.T && col < a.d;
                hraw[q] = load_stream<uint16_t, 8, kNtLoad>(ok ? h0 + 16 * q * plane : hbase);
            }
        };
        auto load_v = [&](int s) {
            const uint16_t *vbase = static_cast<const uint16_t *>(a.V) + n * a.d;
            const uint16_t *v0 = vbase + (size_t)(unsigned)src * plane + s * kAllSlab + 8 * ks;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = s * kAllSlab + 32 * u + 8 * ks;
                const bool ok = src < a.S && c < a.d;
                vraw[u] = load_stream<uint16_t, 8, false>(ok ? v0 + 32 * u : vbase);
            }
        };
        load_dh(0);
        load_v(0);

        lds_barrier();  // the previous token's LDS reads are done
        // The per-token phases (weights; softmax and key gradients) issue at
        // a higher wave priority than the slab streams, so that when the two
        // workgroups of a CU are in different phases the short serial chains
        // go first and the streams fill in behind them (measured 1-2% faster
        // than one priority throughout).
        __builtin_amdgcn_s_setprio(1);
        all_site_weights<uint16_t, RP, true>(a, n, alpha, rho, keys, kown, qs);

        // alpha^T operands of this wave's sources (lane (lc, ks): alpha[32 kg +
        // 8 ks + e][src] as hi + lo bf16) and the weights at this lane's G
        // entries; alpha's LDS then holds the key-column gradients.
        bf16x8_t Ahi[KG], Alo[KG];
        float av[MT][4];
#pragma unroll
        for (int kg = 0; kg < KG; ++kg) {
            float w8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                w8[e] = alpha[(32 * kg + 8 * ks + e) * kAlphaRow + src];
            u32x4_t hi, lo;
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const unsigned hw = pack_bf16x2(w8[2 * h], w8[2 * h + 1]);
                hi[h] = hw;
                lo[h] = pack_bf16x2(w8[2 * h] - bf16_lo(hw), w8[2 * h + 1] - bf16_hi(hw));
            }
            Ahi[kg] = __builtin_bit_cast(bf16x8_t, hi);
            Alo[kg] = __builtin_bit_cast(bf16x8_t, lo);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                av[mt][e] = alpha[(16 * mt + 4 * ks + e) * kAlphaRow + src];

        f32x4_t G[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            G[mt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        __builtin_amdgcn_s_setprio(0);
        for (int s = 0; s < nslab; ++s) {
            per_lane(lc);
            per_lane(ks);
            per_lane(src);
            per_lane(hch);
            per_lane(hr0);
            unsigned char *buf = dhbuf + (s & 1) * kDhBufBytes;
            // Rows past T, and rows 16 MT .. 32 KG - 1 that the last site
            // group's dV MFMAs read with weight 0, are written as zeros (the
            // buffers hold ds / rho between tokens).
#pragma unroll
            for (int q = 0; q < 2 * KG; ++q) {
                const bool ok = q < MT && hr0 + 16 * q < a.T && s * kAllSlab + 8 * hch < a.d;
                *reinterpret_cast<u32x4_t *>(buf + dh_chunk(hr0 + 16 * q, hch)) =
                    ok ? hraw[q < MT ? q : 0] : u32x4_t{0u, 0u, 0u, 0u};
            }
            if (s + 1 < nslab)
                load_dh(s + 1);
            lds_barrier();
            // G[16 mt + 4 ks + e][src] over this slab's columns.  With more
            // than two key tiles (r > 32) the LDS reads of the A operands go
            // out two column groups at a time ahead of their MFMAs (1-3%
            // faster there); with fewer, that was 1% slower, and each read
            // goes just ahead of its MFMA.
            if constexpr (RT >= 3) {
                constexpr int GB = 2;
#pragma unroll
                for (int u0 = 0; u0 < 4; u0 += GB) {
                    bf16x8_t A[GB][MT];
#pragma unroll
                    for (int u = 0; u < GB; ++u)
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt)
                            A[u][mt] = *reinterpret_cast<const bf16x8_t *>(
                                buf + dh_chunk(16 * mt + lc, 4 * (u0 + u) + ks));
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int u = 0; u < GB; ++u) {
                        const int c = s * kAllSlab + 32 * (u0 + u) + 8 * ks;
                        const bool ok = src < a.S && c < a.d;
                        const bf16x8_t B = __builtin_bit_cast(
                            bf16x8_t, ok ? vraw[u0 + u] : u32x4_t{0u, 0u, 0u, 0u});
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt)
                            G[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[u][mt], B, G[mt],
                                                                            0, 0, 0);
                    }
                }
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const bool ok = src < a.S && s * kAllSlab + 32 * u + 8 * ks < a.d;
                    const bf16x8_t B =
                        __builtin_bit_cast(bf16x8_t, ok ? vraw[u] : u32x4_t{0u, 0u, 0u, 0u});
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const bf16x8_t A = *reinterpret_cast<const bf16x8_t *>(
                            buf + dh_chunk(16 * mt + lc, 4 * u + ks));
                        G[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, G[mt], 0, 0, 0);
                    }
                }
            }
            if (s + 1 < nslab)
                load_v(s + 1);

            // dV: acc[p] holds sources 16 wave + 4 ks + e at column c0 + p.
            f32x4_t acc[8];
#pragma unroll
            for (int p = 0; p < 8; ++p)
                acc[p] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int kg = 0; kg < KG; ++kg) {
                u32x4_t w[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    w[e] = *reinterpret_cast<const u32x4_t *>(buf +
                                                              dh_chunk(32 * kg + 8 * ks + e, lc));
#pragma unroll
                for (int p = 0; p < 8; ++p) {
                    u32x4_t bq;
#pragma unroll
                    for (int h = 0; h < 4; ++h)
                        bq[h] = (p & 1) ? hi_pair(w[2 * h][p / 2], w[2 * h + 1][p / 2])
                                        : lo_pair(w[2 * h][p / 2], w[2 * h + 1][p / 2]);
                    const bf16x8_t B = __builtin_bit_cast(bf16x8_t, bq);
                    acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ahi[kg], B, acc[p], 0, 0, 0);
                    acc[p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Alo[kg], B, acc[p], 0, 0, 0);
                }
            }
            const int c0 = s * kAllSlab + 8 * lc;
            if (c0 < tail0) {
                // Rounded and stored (added to the stored value when accumulating).
                uint16_t *d0 = b.dV + (size_t)(unsigned)(16 * wave + 4 * ks) * plane + n * a.d + c0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = 16 * wave + 4 * ks + e;
                    if (i >= a.S)
                        continue;
                    float v[8];
#pragma unroll
                    for (int p = 0; p < 8; ++p)
                        v[p] = acc[p][e];
                    uint16_t *dst = d0 + e * plane;
                    if (ACC) {
                        float old[8];
                        widen(load_raw<uint16_t, 8>(dst), old);
#pragma unroll
                        for (int p = 0; p < 8; ++p)
                            v[p] += old[p];
                    }
                    u32x4_t o;
#pragma unroll
                    for (int h = 0; h < 4; ++h)
                        o[h] = pack_bf16x2(v[2 * h], v[2 * h + 1]);
                    store_stream<uint16_t, 8, kNtStore>(dst, o);
                }
            } else if (c0 < a.d) {
                // Key columns: kept in fp32 until the key gradient is known.
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float *t = tailbuf + (4 * ks + e) * kTailRow + (c0 - tail0);
                    *reinterpret_cast<f32x4_t *>(t) =
                        f32x4_t{acc[0][e], acc[1][e], acc[2][e], acc[3][e]};
                    *reinterpret_cast<f32x4_t *>(t + 4) =
                        f32x4_t{acc[4][e], acc[5][e], acc[6][e], acc[7][e]};
                }
            }
        }

        if (n + gridDim.x < a.N)
            load_site_keys<RP>(a, n + gridDim.x, kown);
        __builtin_amdgcn_s_setprio(1);

        // Softmax gradient.  Lane (lc, ks) holds G[site 16 mt + 4 ks + e][src].
        float ds[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int site = 16 * mt + 4 * ks + e;
                const float t = row16_sum(av[mt][e] * G[mt][e]);
                if (lc == 0)
                    gpart[wave * kAllMaxSources + site] = t;
            }
        lds_barrier();  // also: every wave is past its last read of the slabs
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int site = 16 * mt + 4 * ks + e;
                float gbar = 0.0f;
#pragma unroll
                for (int w = 0; w < kWaves; ++w)
                    gbar += gpart[w * kAllMaxSources + site];
                ds[mt][e] = av[mt][e] * (G[mt][e] - gbar);
            }
        {
            // ds / rho for dQ, in the slab buffers.
            const float inv = src < a.S ? 1.0f / rho[src] : 0.0f;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    dsr[(16 * mt + 4 * ks + e) * kAlphaRow + src] = ds[mt][e] * inv;
        }

        // u_i = sum_j ds[j][i] Q_j over site groups of 32: the MFMA's k
        // index 8 ks + e stands for site 16 (2 kg + e / 4) + 4 ks + e mod 4 on
        // both operands, so the A operand is this lane's ds as it stands.
        f32x4_t uk[RT];
#pragma unroll
        for (int ct = 0; ct < RT; ++ct)
            uk[ct] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int kg = 0; kg < KG; ++kg) {
            float dv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                dv[e] = 2 * kg + e / 4 < MT ? ds[(2 * kg + e / 4) % MT][e % 4] : 0.0f;
            bf16x8_t Dhi, Dlo;
            split_hilo(dv, Dhi, Dlo);
#pragma unroll
            for (int ct = 0; ct < RT; ++ct) {
                __builtin_amdgcn_sched_barrier(0);
                const int c = 16 * ct + lc;
                // Q[site][c] for sites 4 ks + (a constant per e): the lane's
                // row is formed once, the rest are uniform steps of r.
                const float *qlane = qs + 4 * ks * a.r + c;
                float qv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int so = 16 * (2 * kg + e / 4) + e % 4;
                    qv[e] = (4 * ks + so < a.T && c < a.r) ? qlane[so * a.r] : 0.0f;
                }
                bf16x8_t Qhi, Qlo;
                split_hilo(qv, Qhi, Qlo);
                uk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Dhi, Qhi, uk[ct], 0, 0, 0);
                uk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Dhi, Qlo, uk[ct], 0, 0, 0);
                uk[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Dlo, Qhi, uk[ct], 0, 0, 0);
            }
        }
        // dk_i = (u_i - k_i (k_i . u_i) / (rho_i^2 r)) / rho_i; lane (lc, ks)
        // holds sources 16 wave + 4 ks + e at key column 16 ct + lc.  Projected
        // keys: stored into dK; sliced: added to the key columns' gradient.
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = 16 * wave + 4 * ks + e;
            float kv[RT], dot = 0.0f;
#pragma unroll
            for (int ct = 0; ct < RT; ++ct) {
                const int c = 16 * ct + lc;
                kv[ct] = c < a.r ? bf16_at(keys + i * kKeyRow + c) : 0.0f;
                dot = fmaf(kv[ct], uk[ct][e], dot);
            }
            dot = row16_sum(dot);
            const float inv = i < a.S ? 1.0f / rho[i] : 0.0f;
            const float scale = dot * inv * inv * inv_r;
#pragma unroll
            for (int ct = 0; ct < RT; ++ct) {
                const int c = 16 * ct + lc;
                const float dk = (uk[ct][e] - kv[ct] * scale) * inv;
                if (i < a.S && c < a.r) {
                    if (b.dK) {
                        uint16_t *dst = b.dK + ((size_t)(unsigned)(16 * wave + 4 * ks) * a.N + n) * a.r +
                                        (size_t)e * a.N * a.r + c;
                        float v = dk;
                        if (ACC)
                            v += bf16_at(dst);
                        *dst = (uint16_t)pack_bf16x2(v, 0.0f);
                    } else {
                        tailbuf[(4 * ks + e) * kTailRow + (a.d - a.r - tail0) + c] += dk;
                    }
                }
            }
        }

        // dQ_j += sum_i (ds[j][i] / rho_i) k_i: wave w takes the sites of tile w.
        lds_barrier();
        // A: ds / rho of site 16 wave + lc at sources 32 kg + 8 ks + e (zero
        // past S); B: the keys of those sources at column 16 ct + lc (zero
        // past S and r in LDS).
        if (wave < MT) {
            const int nkg = (a.S + 31) / 32;
#pragma unroll 1
            for (int kg = 0; kg < nkg; ++kg) {
                const float *ar = dsr + (16 * wave + lc) * kAlphaRow + 32 * kg + 8 * ks;
                const f32x4_t a0 = *reinterpret_cast<const f32x4_t *>(ar);
                const f32x4_t a1 = *reinterpret_cast<const f32x4_t *>(ar + 4);
                const float av8[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                bf16x8_t Ahi, Alo;
                split_hilo(av8, Ahi, Alo);
#pragma unroll
                for (int ct = 0; ct < RT; ++ct) {
                    const int c = 16 * ct + lc;
                    u32x4_t kb;
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const uint16_t *k0 = keys + (32 * kg + 8 * ks + 2 * h) * kKeyRow + c;
                        kb[h] = (unsigned)k0[0] | ((unsigned)k0[kKeyRow] << 16);
                    }
                    const bf16x8_t B = __builtin_bit_cast(bf16x8_t, kb);
                    dq[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ahi, B, dq[ct], 0, 0, 0);
                    dq[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Alo, B, dq[ct], 0, 0, 0);
                }
            }
        }

        // Sliced keys: the key columns, value and key gradients together.
        // This wave's 16 sources x (d - tail0) / 8 octets, two per lane.
        if (b.sliced) {
            wave_lds_sync();
            const int noct = (a.d - tail0) / 8;
            for (int f = lane; f < 16 * noct; f += kWaveSize) {
                const int li = f / noct, oc = f % noct;
                const int i = 16 * wave + li;
                if (i >= a.S)
                    continue;
                const float *t = tailbuf + li * kTailRow + 8 * oc;
                const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(t);
                const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(t + 4);
                float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
                uint16_t *dst = b.dV + i * plane + n * a.d + tail0 + 8 * oc;
                if (ACC) {
                    float old[8];
                    widen(load_raw<uint16_t, 8>(dst), old);
#pragma unroll
                    for (int p = 0; p < 8; ++p)
                        v[p] += old[p];
                }
                u32x4_t o;
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    o[h] = pack_bf16x2(v[2 * h], v[2 * h + 1]);
                store_stream<uint16_t, 8, kNtStore>(dst, o);
            }
        }
    }

    if (wave < MT) {
        const int lc = (tid0 % kWaveSize) & 15, ks = (tid0 % kWaveSize) >> 4;
        float *part = b.partial + (size_t)blockIdx.x * b.f.T * b.f.r;
#pragma unroll
        for (int ct = 0; ct < RT; ++ct)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int site = 16 * wave + 4 * ks + e, c = 16 * ct + lc;
                if (site < b.f.T && c < b.f.r)
                    part[site * b.f.r + c] = dq[ct][e];
            }
    }
}

template <int MT, int RT, bool ACC>
void launch_all_bwd_t(const AllBwdArgs &b, unsigned grid, hipStream_t st)
{
    hipLaunchKernelGGL((route_all_bwd_bf16<MT, RT, ACC>), dim3(grid), dim3(kBlock), 0, st, b);
}

template <int MT, bool ACC>
void launch_all_bwd_mt(const AllBwdArgs &b, unsigned grid, hipStream_t st)
{
    switch ((b.f.r + 15) / 16) {
    case 1: launch_all_bwd_t<MT, 1, ACC>(b, grid, st); break;
    case 2: launch_all_bwd_t<MT, 2, ACC>(b, grid, st); break;
    case 3: launch_all_bwd_t<MT, 3, ACC>(b, grid, st); break;
    default: launch_all_bwd_t<MT, 4, ACC>(b, grid, st); break;
    }
}

template <bool ACC>
void launch_all_bwd_acc(const AllBwdArgs &b, unsigned grid, hipStream_t st)
{
    switch ((b.f.T + 15) / 16) {
    case 1: launch_all_bwd_mt<1, ACC>(b, grid, st); break;
    case 2: launch_all_bwd_mt<2, ACC>(b, grid, st); break;
    case 3: launch_all_bwd_mt<3, ACC>(b, grid, st); break;
    default: launch_all_bwd_mt<4, ACC>(b, grid, st); break;
    }
}

}  // namespace

int64_t all_bwd_workgroups(int64_t N) { return N < kAllBwdGrid ? N : kAllBwdGrid; }

namespace {

// The fused backward takes bf16 storage and what the fused forward takes.
bool all_bwd_fused(const AllProblem &p) { return p.dtype == LRAR_DTYPE_BF16 && all_fused(p); }

__global__ void __launch_bounds__(256) fill_zero16(u32x4_t *__restrict__ p, size_t n)
{
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        p[i] = u32x4_t{0u, 0u, 0u, 0u};
}

__global__ void __launch_bounds__(256) fill_zero2(uint16_t *__restrict__ p, size_t n)
{
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        p[i] = 0;
}

// Zeros `bytes` (even) bytes at p with a kernel (no memset node, so a
// captured graph replays it like any other launch).
hipError_t launch_zero(void *p, size_t bytes, hipStream_t st)
{
    if (!p || bytes == 0)
        return hipSuccess;
    if (reinterpret_cast<uintptr_t>(p) % 16 == 0 && bytes % 16 == 0) {
        const size_t n = bytes / 16;
        const unsigned grid = (unsigned)std::min<size_t>((n + 255) / 256, 8192);
        hipLaunchKernelGGL(fill_zero16, dim3(grid), dim3(256), 0, st, static_cast<u32x4_t *>(p),
                           n);
    } else {
        const size_t n = bytes / 2;
        const unsigned grid = (unsigned)std::min<size_t>((n + 255) / 256, 8192);
        hipLaunchKernelGGL(fill_zero2, dim3(grid), dim3(256), 0, st, static_cast<uint16_t *>(p),
                           n);
    }
    return hipGetLastError();
}

}  // namespace

size_t all_bwd_workspace_bytes(const AllProblem &p)
{
    if (!all_bwd_fused(p))
        return bwd_workspace_bytes(all_site_problem(p, p.T - 1));
    return (size_t)all_bwd_workgroups(p.N) * (size_t)p.T * (size_t)p.r * sizeof(float);
}

int check_all_bwd_supported(const AllProblem &p, std::string *why)
{
    if (p.N > ((int64_t)1 << 30)) {
        *why = "N above 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if (all_bwd_fused(p))
        return LRAR_OK;
    // Full-rank keys, fp32 storage, or more than 64 sources, sites or key
    // columns: site by site, each site's accumulating single-site backward.
    std::string w;
    if (check_supported(all_site_problem(p, p.T - 1), true, &w) != LRAR_OK) {
        *why = "all-sites backward, site by site: " + w;
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_all_bwd(const AllProblem &p, const void *dH, void *dV, void *dK, float *dQ, void *ws,
                   bool accumulate, hipStream_t st, std::string *err)
{
    if (!all_bwd_fused(p)) {
        // Site by site: each site's backward adds into the gradients of its
        // prefix and into its row of dQ, after one zero fill when overwriting.
        const size_t es = p.dtype == LRAR_DTYPE_BF16 ? 2 : 4;
        if (!accumulate) {
            hipError_t e = launch_zero(dV, (size_t)p.S * p.N * p.d * es, st);
            if (e == hipSuccess && p.mode == LRAR_MODE_PROJECTED)
                e = launch_zero(dK, (size_t)p.S * p.N * p.r * es, st);
            if (e == hipSuccess)
                e = launch_zero(dQ, (size_t)p.T * p.r * sizeof(float), st);
            if (e != hipSuccess)
                return hip_status(e, "route_all_bwd zero fill", err);
        }
        for (int64_t j = 0; j < p.T; ++j) {
            const int rc = launch_bwd(all_site_problem(p, j),
                                      static_cast<const char *>(dH) + (size_t)j * p.N * p.d * es,
                                      dV, dK, dQ + j * p.r, ws, true, st, err);
            if (rc != LRAR_OK)
                return rc;
        }
        return LRAR_OK;
    }
    const unsigned grid = (unsigned)all_bwd_workgroups(p.N);
    float *partial = static_cast<float *>(ws);
    if (grid > 0) {
        AllBwdArgs b;
        b.f.V = p.V;
        b.f.keys = p.mode == LRAR_MODE_PROJECTED ? p.K : p.V;
        b.f.Q = p.Q;
        b.f.H = nullptr;
        b.f.neff = nullptr;
        b.f.S = (int)p.S;
        b.f.d = (int)p.d;
        b.f.r = (int)p.r;
        b.f.krow = p.mode == LRAR_MODE_PROJECTED ? (int)p.r : (int)p.d;
        b.f.koff = p.mode == LRAR_MODE_PROJECTED ? 0 : (int)(p.d - p.r);
        b.f.first = (int)p.first;
        b.f.T = (int)p.T;
        b.f.N = p.N;
        b.f.eps = p.eps;
        b.f.kvec = b.f.r % 8 == 0 && b.f.koff % 8 == 0 && b.f.krow % 8 == 0 &&
                   reinterpret_cast<uintptr_t>(b.f.keys) % 16 == 0;
        b.dH = static_cast<const uint16_t *>(dH);
        b.dV = static_cast<uint16_t *>(dV);
        b.dK = static_cast<uint16_t *>(dK);
        b.partial = partial;
        b.sliced = p.mode == LRAR_MODE_SLICED;
        if (accumulate)
            launch_all_bwd_acc<true>(b, grid, st);
        else
            launch_all_bwd_acc<false>(b, grid, st);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return hip_status(e, "route_all_bwd", err);
    }
    return hip_status(launch_dq_reduce(partial, dQ, (int)grid, (int)(p.T * p.r), accumulate, st),
                      "route_all_bwd dq reduction", err);
}

}  // namespace lrar
