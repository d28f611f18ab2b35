// Every read site of a pass over one source stack in one launch (Sec. 3.1,
// Eq. full_attnres_source_set: site t reads the sources 0 .. t-1), with the
// low-rank keys of Sec. 3.2-3.4 and, optionally, each site's effective
// number of sources (Sec. 4.5, Eq. effective_sources).
//
// Site j = 0 .. T-1 reads the first first+j sources.  Once every o_i of a
// pass exists (recomputing the routed states in the backward, probing a
// trained model), the T sites can share one read of the stack: per token the
// routed states of all sites are one small dense product
//     Hn[T][d] = An[T][S] * On[S][d],   An[j][i] = alpha_{j,i} (0 past the
// site's prefix), On = the token's S source rows,
// which this kernel evaluates on the matrix cores.  The stack is read once
// instead of once per site (sum_j (first+j) row reads), and H is written
// once.
//
// One workgroup (4 waves) per token:
//   1. wave w scores the 16 sites of tile w against every source on the
//      matrix cores (s_{j,i} rho_i = Q_j . k_i, Eqs. lr_key_norm and
//      lr_attnres_weight; rho_i from the same key loads), takes each site's
//      softmax over its prefix with lane exchanges, writes alpha to LDS
//      (zero past the prefix) and N_eff, which follows from the same sums:
//          -sum alpha_i log alpha_i = log z - sum alpha_i (s_i - m);
//   2. each wave takes 128-column slabs of the row.  Lane l owns 8
//      consecutive columns c0 = 128 slab + 8 (l mod 16) and loads them from
//      the sources of its k-slice with 16-byte reads; an MFMA's column index
//      l mod 16 then stands for column c0 + p in the p-th of 8 MFMAs, so the
//      loaded vectors feed the matrix cores without an LDS transpose and
//      the outputs come back as 8 consecutive columns per lane.
// bf16 storage: v_mfma_f32_16x16x32_bf16 over 32 sources per step; alpha
// enters as a pair of bf16 (hi = RNE(alpha), lo = RNE(alpha - hi), relative
// error <= 2^-17), two MFMAs per tile, fp32 accumulation: the products with
// the bf16 values are exact, so the state keeps fp32-level accuracy.
// fp32 storage: v_mfma_f32_16x16x4_f32 over 4 sources per step, alpha and
// the values as they are.
// Sources past a site's prefix enter its product with weight exactly 0.
#include "route_all_weights.h"

#include <algorithm>

namespace lrar {

namespace {

constexpr int kAllFwdGrid = 256;  // persistent workgroups above 48 sites (one per CU)

// Largest prefix read by a site of tile mt (sites 16 mt .. 16 mt + 15).
__device__ __forceinline__ int tile_prefix(const AllArgs &a, int mt)
{
    return a.first + min(16 * mt + 15, a.T - 1);
}

// Issue the loads of the lane's 8 sources of group kg (sources 32 kg + 8 ks
// + e) at columns c0 .. c0 + 7.  Lanes past the columns or the sources load
// nothing; their entries are masked to zero when the B operands are built.
__device__ __forceinline__ void load_group(const uint16_t *__restrict__ vrow, size_t plane,
                                           int S, int kg, int ks, bool ok, u32x4_t (&raw)[8])
{
    // One 64-bit row address per lane; the other sources are whole planes on.
    const uint16_t *r0 = vrow + (size_t)(unsigned)(32 * kg + 8 * ks) * plane;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int i = 32 * kg + 8 * ks + e;
        if (ok && i < S)
            raw[e] = load_stream<uint16_t, 8, kNtLoad>(r0 + e * plane);
    }
}

// bf16 storage: 32 sources per MFMA step, at most 2 steps (S <= 64).  One
// source group is in flight while the previous one is multiplied; the first
// is issued before the weights are computed.  Every site tile multiplies
// every group: the weights past a site's prefix are zero, and skipping the
// few empty tile-group pairs would cost more in register traffic than the
// matrix cores save.  One token: with PERSIST, its keys come in kown and
// the next token's keys (token nnext) are loaded into kown once its
// weights are formed, so that they arrive during its mix.
template <int MT, int RP, bool PERSIST>
__device__ __forceinline__ void all_fwd_token(const AllArgs &a, int64_t n, float *alpha,
                                              u32x4_t *kown, int64_t nnext)
{
    const int lane = threadIdx.x % kWaveSize, wave = threadIdx.x / kWaveSize;
    const int col = lane & 15, ks = lane >> 4;
    const uint16_t *V = static_cast<const uint16_t *>(a.V) + n * a.d + 8 * col;
    uint16_t *H = static_cast<uint16_t *>(a.H) + n * a.d + 8 * col;
    const size_t plane = (size_t)a.N * a.d;
    const int ngroups = (a.S + 31) / 32;
    const int nslab = (a.d + kAllSlab - 1) / kAllSlab;

    u32x4_t raw[8];
    if (wave < nslab)
        load_group(V + wave * kAllSlab, plane, a.S, 0, ks, wave * kAllSlab + 8 * col < a.d, raw);
    if constexpr (PERSIST) {
        lds_barrier();  // every wave is done with the previous token's weights
        all_site_weights<uint16_t, RP>(a, n, alpha, nullptr, nullptr, kown);
        if (nnext < a.N)
            load_site_keys<RP>(a, nnext, kown);
    } else {
        all_site_weights<uint16_t, RP>(a, n, alpha);
    }

    for (int slab = wave; slab < nslab; slab += kWaves) {
        const int c0 = slab * kAllSlab + 8 * col;
        const bool ok = c0 < a.d;
        f32x4_t acc[MT][8];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int p = 0; p < 8; ++p)
                acc[mt][p] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        for (int kg = 0; kg < ngroups; ++kg) {
            // B operands: column c0 + p of the lane's 8 sources, as bf16 pairs.
            unsigned w[8][4];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const bool v = ok && 32 * kg + 8 * ks + e < a.S;
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    w[e][h] = v ? raw[e][h] : 0u;
            }
            u32x4_t b[8];
#pragma unroll
            for (int p = 0; p < 8; ++p)
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    b[p][h] = (p & 1) ? hi_pair(w[2 * h][p / 2], w[2 * h + 1][p / 2])
                                      : lo_pair(w[2 * h][p / 2], w[2 * h + 1][p / 2]);
            // Prefetch: the next group of this slab, else group 0 of the next.
            int ns = slab, nk = kg + 1;
            if (nk == ngroups) {
                nk = 0;
                ns += kWaves;
            }
            if (ns < nslab)
                load_group(V + ns * kAllSlab, plane, a.S, nk, ks, ns * kAllSlab + 8 * col < a.d,
                           raw);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const float *ar = alpha + (16 * mt + col) * kAlphaRow + 32 * kg + 8 * ks;
                const f32x4_t a0 = *reinterpret_cast<const f32x4_t *>(ar);
                const f32x4_t a1 = *reinterpret_cast<const f32x4_t *>(ar + 4);
                const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                u32x4_t ahi, alo;
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const unsigned hw = pack_bf16x2(av[2 * h], av[2 * h + 1]);
                    ahi[h] = hw;
                    alo[h] = pack_bf16x2(av[2 * h] - bf16_lo(hw), av[2 * h + 1] - bf16_hi(hw));
                }
                const bf16x8_t A_hi = __builtin_bit_cast(bf16x8_t, ahi);
                const bf16x8_t A_lo = __builtin_bit_cast(bf16x8_t, alo);
#pragma unroll
                for (int p = 0; p < 8; ++p) {
                    const bf16x8_t B = __builtin_bit_cast(bf16x8_t, b[p]);
                    acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A_hi, B, acc[mt][p], 0, 0, 0);
                    acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A_lo, B, acc[mt][p], 0, 0, 0);
                }
            }
        }
        // Lane l holds sites 16 mt + 4 (l / 16) + e, columns c0 .. c0 + 7.
        if (ok) {
            uint16_t *h0 = H + (size_t)(unsigned)(4 * ks) * plane + slab * kAllSlab;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int site = 16 * mt + 4 * ks + e;
                    if (site < a.T) {
                        u32x4_t o;
#pragma unroll
                        for (int h = 0; h < 4; ++h)
                            o[h] = pack_bf16x2(acc[mt][2 * h][e], acc[mt][2 * h + 1][e]);
                        store_stream<uint16_t, 8, kNtStore>(h0 + (16 * mt + e) * plane, o);
                    }
                }
        }
    }
}

// Up to 48 sites, two or more workgroups per CU, one token each: the
// workgroups cover each other's key loads.  Above 48 sites a workgroup
// fills its CU, so it is persistent over a stride of tokens and loads the
// next token's keys during the current token's mix (17% faster at 63
// sites; at 48 sites the same form is 2-7% slower).
template <int MT, int RP>
__global__ __launch_bounds__(kBlock, MT <= 3 ? 2 : 1) void route_all_fwd_bf16(AllArgs a)
{
    __shared__ __align__(16) float alpha[kAllMaxSources * kAlphaRow];
    if constexpr (MT <= 3) {
        all_fwd_token<MT, RP, false>(a, blockIdx.x, alpha, nullptr, 0);
    } else {
        u32x4_t kown[4 * (RP / 32)];
        if (blockIdx.x < a.N)
            load_site_keys<RP>(a, blockIdx.x, kown);
        for (int64_t n = blockIdx.x; n < a.N; n += gridDim.x)
            all_fwd_token<MT, RP, true>(a, n, alpha, kown, n + gridDim.x);
    }
}

// fp32 storage: 4 sources per MFMA step.
template <int MT, int RP>
__global__ __launch_bounds__(kBlock) void route_all_fwd_f32(AllArgs a)
{
    __shared__ __align__(16) float alpha[kAllMaxSources * kAlphaRow];
    const int64_t n = blockIdx.x;
    all_site_weights<float, RP>(a, n, alpha);

    const int lane = threadIdx.x % kWaveSize, wave = threadIdx.x / kWaveSize;
    const int col = lane & 15, ks = lane >> 4;
    const float *V = static_cast<const float *>(a.V);
    float *H = static_cast<float *>(a.H);
    const size_t plane = (size_t)a.N * a.d;
    const int nslab = (a.d + kAllSlab - 1) / kAllSlab;

    for (int slab = wave; slab < nslab; slab += kWaves) {
        const int c0 = slab * kAllSlab + 8 * col;
        const bool ok = c0 < a.d;
        f32x4_t acc[MT][8];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int p = 0; p < 8; ++p)
                acc[mt][p] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        for (int i0 = 0; i0 < a.S; i0 += 4) {
            const int i = i0 + ks;
            f32x4_t v0 = {0.0f, 0.0f, 0.0f, 0.0f}, v1 = v0;
            if (ok && i < a.S) {
                const float *src = V + i * plane + n * a.d + c0;
                v0 = load_stream<float, 4, kNtLoad>(src);
                v1 = load_stream<float, 4, kNtLoad>(src + 4);
            }
            const float bv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                if (i0 >= tile_prefix(a, mt))
                    continue;
                const float A = alpha[(16 * mt + col) * kAlphaRow + i];
#pragma unroll
                for (int p = 0; p < 8; ++p)
                    acc[mt][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(A, bv[p], acc[mt][p], 0, 0, 0);
            }
        }
        if (ok) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int site = 16 * mt + 4 * ks + e;
                    if (site < a.T) {
                        float *dst = H + site * plane + n * a.d + c0;
                        store_stream<float, 4, kNtStore>(
                            dst, f32x4_t{acc[mt][0][e], acc[mt][1][e], acc[mt][2][e], acc[mt][3][e]});
                        store_stream<float, 4, kNtStore>(
                            dst + 4, f32x4_t{acc[mt][4][e], acc[mt][5][e], acc[mt][6][e], acc[mt][7][e]});
                    }
                }
        }
    }
}

template <int MT, int RP>
hipError_t launch_all_mt_rp(const AllArgs &a, int dtype, hipStream_t st)
{
    if (dtype == LRAR_DTYPE_BF16) {
        // Persistent above 48 sites: one workgroup per CU.
        const unsigned grid = MT <= 3 ? (unsigned)a.N : (unsigned)std::min<int64_t>(a.N, kAllFwdGrid);
        hipLaunchKernelGGL((route_all_fwd_bf16<MT, RP>), dim3(grid), dim3(kBlock), 0, st, a);
    } else {
        hipLaunchKernelGGL((route_all_fwd_f32<MT, RP>), dim3((unsigned)a.N), dim3(kBlock), 0, st, a);
    }
    return hipGetLastError();
}

template <int MT>
hipError_t launch_all_mt(const AllArgs &a, int dtype, hipStream_t st)
{
    if (a.r <= 32)
        return launch_all_mt_rp<MT, 32>(a, dtype, st);
    return launch_all_mt_rp<MT, 64>(a, dtype, st);
}

// Effective number of sources of one site (Sec. 4.5, Eq. effective_sources)
// from the keys alone: one wave per token scores its S sources, then
//     N_eff = exp(-sum alpha_i log alpha_i) = z exp(-t / z),
//     z = sum_i exp(s_i - m),  t = sum_i exp(s_i - m) (s_i - m).
// Full-rank keys run as sliced keys with r = d (Sec. 3.4).
template <typename T, int VEC>
__global__ __launch_bounds__(kBlock) void route_neff(const T *__restrict__ keys,
                                                     const float *__restrict__ q,
                                                     float *__restrict__ neff, int S, int N,
                                                     int r, int krow, int koff, float eps,
                                                     int s_pad)
{
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const int n = blockIdx.x * kWaves + wave;
    if (n >= N)
        return;  // wave-uniform; no workgroup barrier
    float *s = lds + wave * s_pad;
    lr_scores<T, VEC>(keys, q, S, N, r, krow, koff, eps, n, lane, s, nullptr);
    float m = -INFINITY;
    for (int i = lane; i < S; i += kWaveSize)
        m = fmaxf(m, s[i]);
    m = wave_max(m);
    float z = 0.0f, t = 0.0f;
    for (int i = lane; i < S; i += kWaveSize) {
        const float x = s[i] - m;
        const float e = expf(x);
        z += e;
        t = fmaf(e, x, t);
    }
    z = wave_sum(z);
    t = wave_sum(t);
    if (lane == 0)
        neff[n] = z * expf(-t / z);
}

}  // namespace

bool all_fused(const AllProblem &p)
{
    return (p.mode == LRAR_MODE_PROJECTED || p.mode == LRAR_MODE_SLICED) &&
           p.S <= kAllMaxSources && p.T <= kAllMaxSources && p.r <= kAllMaxRank && p.d % 8 == 0;
}

Problem all_site_problem(const AllProblem &p, int64_t j)
{
    return Problem{p.V, p.K, p.Q + j * p.r, p.first + j, p.N, p.d, p.r, p.mode, p.dtype, p.eps,
                   p.dtype};
}

int check_all_supported(const AllProblem &p, std::string *why)
{
    if (p.N > ((int64_t)1 << 30)) {
        *why = "N above 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if (all_fused(p))
        return LRAR_OK;
    // Full-rank keys, or more than 64 sources, sites or key columns: site by
    // site, each site as the single-site forward over its prefix.  The last
    // site reads the most sources and binds.
    std::string w;
    if (check_supported(all_site_problem(p, p.T - 1), false, &w) != LRAR_OK) {
        *why = "all-sites routing, site by site: " + w;
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_all_fwd(const AllProblem &p, hipStream_t st, std::string *err)
{
    if (p.N == 0)
        return LRAR_OK;
    if (!all_fused(p)) {
        // One launch of the single-site forward (and N_eff) per site.
        const size_t es = p.dtype == LRAR_DTYPE_BF16 ? 2 : 4;
        for (int64_t j = 0; j < p.T; ++j) {
            const Problem ps = all_site_problem(p, j);
            int rc = launch_fwd(ps, static_cast<char *>(p.H) + (size_t)j * p.N * p.d * es, st,
                                err);
            if (rc == LRAR_OK && p.neff) {
                // Full rank: the key is the whole value, sliced keys with r = d.
                Problem pn = ps;
                if (pn.mode == LRAR_MODE_FULL)
                    pn.mode = LRAR_MODE_SLICED;
                rc = launch_neff(pn, p.neff + j * p.N, st, err);
            }
            if (rc != LRAR_OK)
                return rc;
        }
        return LRAR_OK;
    }
    AllArgs a;
    a.V = p.V;
    a.keys = p.mode == LRAR_MODE_PROJECTED ? p.K : p.V;
    a.Q = p.Q;
    a.H = p.H;
    a.neff = p.neff;
    a.S = (int)p.S;
    a.d = (int)p.d;
    a.r = (int)p.r;
    a.krow = p.mode == LRAR_MODE_PROJECTED ? (int)p.r : (int)p.d;
    a.koff = p.mode == LRAR_MODE_PROJECTED ? 0 : (int)(p.d - p.r);
    a.first = (int)p.first;
    a.T = (int)p.T;
    a.N = p.N;
    a.eps = p.eps;
    a.kvec = a.r % 8 == 0 && a.koff % 8 == 0 && a.krow % 8 == 0 &&
             reinterpret_cast<uintptr_t>(a.keys) % 16 == 0;
    hipError_t e;
    switch ((a.T + 15) / 16) {
    case 1: e = launch_all_mt<1>(a, p.dtype, st); break;
    case 2: e = launch_all_mt<2>(a, p.dtype, st); break;
    case 3: e = launch_all_mt<3>(a, p.dtype, st); break;
    default: e = launch_all_mt<4>(a, p.dtype, st); break;
    }
    return hip_status(e, "route_all_fwd", err);
}

}  // namespace lrar

namespace lrar {

int launch_neff(const Problem &p, float *neff, hipStream_t st, std::string *err)
{
    if (p.S > 1024) {
        *err = "the effective number of sources supports S <= 1024";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N > ((int64_t)1 << 30)) {
        *err = "N above 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N == 0)
        return LRAR_OK;
    const bool proj = p.mode == LRAR_MODE_PROJECTED;
    const void *keys = proj ? p.K : p.V;
    const int krow = proj ? (int)p.r : (int)p.d;
    const int koff = proj ? 0 : (int)(p.d - p.r);
    const int s_pad = (int)((p.S + 3) / 4 * 4);
    const dim3 grid((unsigned)((p.N + kWaves - 1) / kWaves));
    const size_t lds = (size_t)kWaves * s_pad * sizeof(float);
    if (p.dtype == LRAR_DTYPE_BF16)
        hipLaunchKernelGGL((route_neff<uint16_t, 8>), grid, dim3(kBlock), lds, st,
                           static_cast<const uint16_t *>(keys), p.q, neff, (int)p.S, (int)p.N,
                           (int)p.r, krow, koff, p.eps, s_pad);
    else
        hipLaunchKernelGGL((route_neff<float, 4>), grid, dim3(kBlock), lds, st,
                           static_cast<const float *>(keys), p.q, neff, (int)p.S, (int)p.N,
                           (int)p.r, krow, koff, p.eps, s_pad);
    return hip_status(hipGetLastError(), "route_neff launch", err);
}

}  // namespace lrar
