// Scores and depth softmax of every read site of a pass for one token, on
// the matrix cores: shared by the all-sites forward and backward.  Internal
// to the library.
#pragma once

#include "route_common.h"

namespace lrar {

constexpr int kAllMaxSources = 64;  // sources S, and sites T
constexpr int kAllMaxRank = 64;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kAllSlab = 128;                     // columns per wave pass
constexpr int kAlphaRow = kAllMaxSources + 4;     // floats per LDS alpha row
constexpr int kKeyRow = kAllMaxRank + 8;          // bf16 per LDS key row

struct AllArgs {
    const void *V;       // [S][N][d]
    const void *keys;    // projected: K [S][N][r]; sliced: V
    const float *Q;      // [T][r]
    void *H;             // [T][N][d]
    float *neff;         // [T][N] or NULL
    int S, d, r, krow, koff, first, T;
    int64_t N;
    float eps;
    bool kvec;           // bf16 keys readable as 16-byte vectors
};

// Scores, softmax and N_eff of one token.  Wave w owns the sites of tile w
// (16 w .. 16 w + 15) and computes their scores against all sources on the
// matrix cores: s_{j,i} rho_i = Q_j . k_i is a [16 x r] x [r x S] product per
// tile.  The MFMA's B operand is the keys as stored (lane l: source
// 16 nt + (l mod 16), key elements kb .. kb + 7 of its k-slice), so rho_i
// comes from the same loads: each lane squares its elements and the four
// k-slices of a source are summed with two exchanges.  The result tile has
// sites on rows 4 (l / 16) + e and sources on column l mod 16, so a site's
// softmax is a reduction over the 16 lanes of its row group.
// Writes alpha (fp32 [64][kAlphaRow], zero past each prefix and for absent
// sites) to LDS and N_eff to global; ends with a workgroup barrier (LDS only).
//
// bf16 storage: v_mfma_f32_16x16x32_bf16, 32 key elements per step; the keys
// are exact in bf16 and Q enters as hi + lo bf16 (two MFMAs), so the dot
// product has fp32-level accuracy.  fp32 storage: v_mfma_f32_16x16x4_f32,
// 4 key elements per step, operands as they are.
//
// SAVE (bf16 storage only): wave 0 also leaves every source's key (bf16,
// [64][kKeyRow], zero past r and past S) and rho_i ([64]) in LDS, for the
// backward's key-path terms.
//
// bf16 storage can take the keys already loaded (kpre, from load_site_keys,
// so that they can be issued ahead of other loads) and the queries from LDS
// (qlds, Q [T][r]); by default both are read here from global memory.
// Sum and maximum over the 16 lanes of each row of the wave, returned to
// all 16: four DPP moves (group_sum / group_max over groups of 16).
__device__ __forceinline__ float row16_sum(float x) { return group_sum(x, 16); }
__device__ __forceinline__ float row16_max(float x) { return group_max(x, 16); }

template <int RP>
__device__ __forceinline__ void load_site_keys(const AllArgs &a, int64_t n, u32x4_t *kraw)
{
    constexpr int KK = RP / 32;
    const int lane = threadIdx.x % kWaveSize;
    const int col = lane & 15, ks = lane >> 4;
    const uint16_t *keys = static_cast<const uint16_t *>(a.keys) + n * a.krow + a.koff;
    const size_t kplane = (size_t)a.N * a.krow;
    if (a.kvec) {
        // Sources past S and elements past r load a valid address; they are
        // zeroed where the keys are used.
        // One 64-bit row address per lane; the other rows are 16 planes on.
        const uint16_t *k0 = keys + (size_t)(unsigned)col * kplane + 8 * ks;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int i = 16 * nt + col, c = 32 * kk + 8 * ks;
                const bool ok = i < a.S && c < a.r;
                kraw[nt * KK + kk] = load_raw<uint16_t, 8>(ok ? k0 + 16 * nt * kplane + 32 * kk : keys);
            }
    } else {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int i = 16 * nt + col, c = 32 * kk + 8 * ks;
                u32x4_t kr = {0u, 0u, 0u, 0u};
                if (i < a.S && c < a.r) {
                    const uint16_t *kp = keys + i * kplane + c;
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        const unsigned x0 = c + 2 * h < a.r ? kp[2 * h] : 0u;
                        const unsigned x1 = c + 2 * h + 1 < a.r ? kp[2 * h + 1] : 0u;
                        kr[h] = x0 | (x1 << 16);
                    }
                }
                kraw[nt * KK + kk] = kr;
            }
    }
}

template <typename T, int RP, bool SAVE = false>
__device__ __forceinline__ void all_site_weights(const AllArgs &a, int64_t n, float *alpha,
                                                 float *rho_out = nullptr,
                                                 uint16_t *key_out = nullptr,
                                                 const u32x4_t *kpre = nullptr,
                                                 const float *qlds = nullptr)
{
    // The lane's indices are formed here, each call, instead of being held
    // across a persistent caller's token loop (where they would take
    // registers for the kernel's lifetime).
    unsigned tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid % kWaveSize, wave = tid / kWaveSize;
    const int col = lane & 15, ks = lane >> 4;
    const int qsite = 16 * wave + col;  // site of this lane's A-operand row
    const T *keys = static_cast<const T *>(a.keys) + n * a.krow + a.koff;
    const size_t kplane = (size_t)a.N * a.krow;

    f32x4_t D[4];
    float ss[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
        D[nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        ss[nt] = 0.0f;
    }
    if constexpr (std::is_same<T, uint16_t>::value) {
        constexpr int KK = RP / 32;
        bf16x8_t Ahi[KK], Alo[KK];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            float qv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int c = 32 * kk + 8 * ks + e;
                qv[e] = (qsite < a.T && c < a.r)
                            ? (qlds ? qlds[qsite * a.r + c] : a.Q[(size_t)qsite * a.r + c])
                            : 0.0f;
            }
            u32x4_t hi, lo;
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const unsigned hw = pack_bf16x2(qv[2 * h], qv[2 * h + 1]);
                hi[h] = hw;
                lo[h] = pack_bf16x2(qv[2 * h] - bf16_lo(hw), qv[2 * h + 1] - bf16_hi(hw));
            }
            Ahi[kk] = __builtin_bit_cast(bf16x8_t, hi);
            Alo[kk] = __builtin_bit_cast(bf16x8_t, lo);
        }
        u32x4_t kown[4 * KK];
        if (!kpre)
            load_site_keys<RP>(a, n, kown);
        const u32x4_t *kraw = kpre ? kpre : kown;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int i = 16 * nt + col;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int c = 32 * kk + 8 * ks;
                const u32x4_t kr = (i < a.S && c < a.r) ? kraw[nt * KK + kk]
                                                        : u32x4_t{0u, 0u, 0u, 0u};
                if (SAVE && wave == 0)
                    *reinterpret_cast<u32x4_t *>(key_out + i * kKeyRow + c) = kr;
                float x[8];
                widen(kr, x);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    ss[nt] = fmaf(x[e], x[e], ss[nt]);
                const bf16x8_t B = __builtin_bit_cast(bf16x8_t, kr);
                D[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ahi[kk], B, D[nt], 0, 0, 0);
                D[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Alo[kk], B, D[nt], 0, 0, 0);
            }
        }
    } else {
        constexpr int KK = RP / 4;
        float A[KK];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const int c = 4 * kk + ks;
            A[kk] = (qsite < a.T && c < a.r) ? a.Q[(size_t)qsite * a.r + c] : 0.0f;
        }
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int i = 16 * nt + col;
#pragma unroll
            for (int kk = 0; kk < KK; ++kk) {
                const int c = 4 * kk + ks;
                const float x = (i < a.S && c < a.r)
                                    ? reinterpret_cast<const float *>(keys)[i * kplane + c]
                                    : 0.0f;
                ss[nt] = fmaf(x, x, ss[nt]);
                D[nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(A[kk], x, D[nt], 0, 0, 0);
            }
        }
    }

    // Scores: lane l holds sites 16 w + 4 (l / 16) + e against sources
    // 16 nt + (l mod 16).
    // One reciprocal per key instead of a division per score.
    float s[4][4];
    float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    const float inv_r = 1.0f / (float)a.r;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
        float t = ss[nt];
        t += __shfl_xor(t, 16, kWaveSize);
        t += __shfl_xor(t, 32, kWaveSize);
        const float rho = sqrtf(fmaf(t, inv_r, a.eps));
        const float irho = 1.0f / rho;
        const int i = 16 * nt + col;
        if (SAVE && wave == 0 && ks == 0)
            rho_out[i] = rho;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int site = 16 * wave + 4 * ks + e;
            const bool v = site < a.T && i < a.first + site;
            s[nt][e] = v ? D[nt][e] * irho : -INFINITY;
            m[e] = fmaxf(m[e], s[nt][e]);
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        m[e] = row16_max(m[e]);
    float ex[4][4], z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            ex[nt][e] = s[nt][e] > -INFINITY ? expf(s[nt][e] - m[e]) : 0.0f;
            z[e] += ex[nt][e];
        }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        z[e] = row16_sum(z[e]);
    float sa[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int site = 16 * wave + 4 * ks + e;
        const float inv = z[e] > 0.0f ? 1.0f / z[e] : 0.0f;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const float al = ex[nt][e] * inv;
            if (ex[nt][e] > 0.0f)
                sa[e] = fmaf(al, s[nt][e] - m[e], sa[e]);
            alpha[site * kAlphaRow + 16 * nt + col] = al;
        }
    }
    if (a.neff) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sa[e] = row16_sum(sa[e]);
            const int site = 16 * wave + 4 * ks + e;
            if (col == 0 && site < a.T)
                a.neff[(size_t)site * a.N + n] = expf(logf(z[e]) - sa[e]);
        }
    }
    lds_barrier();
}

// Pairs of bf16 from two packed words: the low halves (lo_pair) or the
// high halves (hi_pair) of x and y, x's in the low half of the result.  An
// 8 x 8 block of bf16 (8 rows of 8 consecutive columns, one 16-byte row per
// register quad) is transposed with these into MFMA operands that hold one
// column of 8 rows.
// Each is one byte permute (v_perm_b32: selector bytes 0-3 pick bytes of the
// second operand, 4-7 of the first).
__device__ __forceinline__ unsigned lo_pair(unsigned x, unsigned y)
{
    return __builtin_amdgcn_perm(y, x, 0x05040100u);  // (x & 0xffff) | (y << 16)
}
__device__ __forceinline__ unsigned hi_pair(unsigned x, unsigned y)
{
    return __builtin_amdgcn_perm(y, x, 0x07060302u);  // (x >> 16) | (y & 0xffff0000)
}

}  // namespace

}  // namespace lrar
