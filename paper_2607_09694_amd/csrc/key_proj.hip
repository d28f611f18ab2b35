// The projected-key producer (Sec. 3.3, Eq. fused_projection): the output
// projection of a residual-writing sub-layer and its key projection are one
// matrix [W^O; W^K] of d + r rows applied to the activation a_n entering the
// output projection, [o_n; k_n] = [W^O; W^K] a_n.  One GEMM
//     C[N][d + r] = A[N][m] * W[d + r][m]^T
// on the matrix cores, whose epilogue writes columns 0 .. d-1 into the value
// slot O[N][d] (the sub-layer's plane of the value stack) and columns
// d .. d+r-1 into the key slot K[N][r] (its plane of the key stack): the
// activation is read once for both, and the key costs r extra output
// columns (about r / d more work) instead of a second pass over A.
//
// Tiling for gfx950: a workgroup of 8 waves (two per SIMD) computes 256
// tokens x up to 288 output columns.  Column tiles are 256 wide, except the
// last, which also takes the remaining columns up to 288: with d a multiple
// of 256 and r <= 32 the key columns ride along with the last value tile,
// and N = 16384 tokens at d = 1024 make exactly 256 workgroups, one per CU.
// Waves are 4 x 2; a wave owns 64 rows and half of the tile's columns, at
// most 9 column tiles of v_mfma_f32_16x16x32_bf16 with fp32 accumulators
// (at most 144 per lane, so two waves fit a SIMD's registers).  Both
// operands are k-contiguous in memory (A row-major, W in the [out][in]
// layout of a linear layer).  64-wide k-slices of both go straight from
// memory to LDS with buffer loads (no register staging), double-buffered:
// the next slice is in flight while the current one feeds the MFMAs.  The
// buffer resources cover only the workgroup's rows, so rows past N or past
// the output read as zero.  LDS rows are 128 bytes with the 16-byte chunks
// XOR-swizzled by (row / 2) mod 8, so that the 16 consecutive rows that one
// MFMA operand read touches fall on distinct banks.  Within a k-step the
// MFMAs go column tile by column tile; the B fragments are read a few
// columns ahead and the next k-step's A fragments during the first columns.
// Workgroups are ordered so that the column tiles of one row tile run on
// one XCD and share its L2 copy of the A slice.  The epilogue rounds to bf16
// (nearest even), stages half of the tile at a time through LDS and writes
// 16-byte row segments, split between O and K at column d.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <string>

#include "route_common.h"

namespace lrar {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kPM = 256;             // tokens per workgroup tile
constexpr int kPN = 256;             // output columns per full column tile
constexpr int kPNMax = kPN + 32;     // the last column tile may reach 288
constexpr int kPK = 64;              // k per LDS stage
constexpr int kRow = kPK * 2;        // bytes per LDS row of a stage (unpadded)
constexpr int kABlocks = kPM / 8;    // 1 KB blocks of 8 rows: A part of a stage
constexpr int kBBlocks = kPNMax / 8; // ... and W part
constexpr int kStageBytes = (kPM + kPNMax) * kRow;
constexpr int kWaves8 = 8;           // waves per workgroup (2 per SIMD)
constexpr int kLoads = (kABlocks + kBBlocks + kWaves8 - 1) / kWaves8;  // direct loads per wave
constexpr int kCd = kPNMax + 8;      // LDS row stride of the output half-tile (elements)
constexpr int kPThreads = kWaves8 * kWaveSize;
// Buffer resource word 3 for raw (untyped) loads on gfx9-family parts.
constexpr int kRawBufferFlags = 0x00020000;

static_assert(kABlocks % kWaves8 == 0, "A blocks split evenly over the waves");
static_assert(2 * kStageBytes >= kPM / 2 * kCd * 2, "output half-tile fits the stages");

struct ProjArgs {
    const uint16_t *A;  // [N][m]
    const uint16_t *W;  // [d + r][m]
    uint16_t *O;        // [N][d] or NULL (d = 0)
    uint16_t *K;        // [N][r] or NULL (r = 0)
    int64_t N;
    int m, d, r, ncol;
    bool ovec, kvec;    // O / K rows writable as 16-byte vectors
};

// Column tiles: ncol - 1 of width 256, the last one the rest (<= 288).
int key_proj_col_tiles(int64_t nout)
{
    return nout <= kPNMax ? 1 : (int)((nout - kPNMax + kPN - 1) / kPN) + 1;
}

// LDS placement of 16-byte chunk c (0..7) of stage row `row`: rows are 128
// bytes, and the chunk is XOR-swizzled with (row / 2) mod 8, so the 16
// consecutive rows that one MFMA operand read touches spread over all banks.
__device__ __forceinline__ int chunk_at(int row, int c) { return row * kRow + 16 * (c ^ ((row >> 1) & 7)); }

// The k loop and epilogue of one workgroup; each wave computes NJ column
// tiles of 16 (compile time, so that no MFMA sits behind a branch).
template <int NJ>
__device__ __forceinline__ void key_proj_tile(const ProjArgs &a, unsigned char *lds, int64_t n0,
                                              int j0, int width, int half)
{
    const int tid = threadIdx.x;
    const int lane = tid % kWaveSize, wave = __builtin_amdgcn_readfirstlane(tid / kWaveSize);
    const int wm = wave >> 1, wn = wave & 1;  // 4 row groups of 64 x 2 column halves
    const int nout = a.d + a.r;
    const int nk = (a.m + kPK - 1) / kPK;

    // Stage kt into LDS buffer `buf` with buffer loads straight to LDS.  The
    // wave's u-th load fills 1 KB block (wave + 4 u), rows 8 blk .. 8 blk + 7:
    // lane l writes bytes 16 l .. 16 l + 15 of the block, i.e. row l / 8,
    // placed chunk l mod 8, which holds global chunk (l mod 8) ^ swizzle.
    // The buffer resources cover the workgroup's rows of A and of W only, so
    // rows past N, past the tile or past d + r read as zero.  A chunk past m
    // reads the next row's first elements; it is zeroed in LDS (zero_tail).
    // Each lane needs one offset; the row group and the k offset are scalar.
    // Block blk = wave + 8 u holds rows 8 blk .. 8 blk + 7 of A (blk < 32) or
    // of W; its swizzle (row / 2) mod 8 = (4 (blk mod 2) + l / 16) mod 8 only
    // depends on the wave's parity, so each lane needs one offset.
    const int rl = 8 * wave + (lane >> 3);             // row within a 64-row group
    const int voff = rl * a.m * 2 + 16 * ((lane & 7) ^ ((rl >> 1) & 7));
    const int arows = (int)min((int64_t)kPM, a.N - n0);
    const int brows = max(0, min(width, nout - j0));
    const __amdgpu_buffer_rsrc_t ares = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.A + n0 * a.m), 0, arows * a.m * 2, kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t bres = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.W + (size_t)j0 * a.m), 0, brows * a.m * 2, kRawBufferFlags);
    auto issue = [&](int kt, int buf) {
        unsigned char *sb = lds + buf * kStageBytes;
        const int kbytes = kt * kPK * 2;
#pragma unroll
        for (int u = 0; u < kLoads; ++u) {
            const int blk = wave + kWaves8 * u;
            if (u < kABlocks / kWaves8)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ares, (lds_void_t *)(sb + 1024 * blk), 16,
                                                         voff, u * 128 * a.m + kbytes, 0, 0);
            else if (blk < kABlocks + kBBlocks)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    bres, (lds_void_t *)(sb + 1024 * blk), 16, voff,
                    (u - kABlocks / kWaves8) * 128 * a.m + kbytes, 0, 0);
        }
    };

    f32x4_t acc[4][NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // Operand fragments: lane l reads row base + l mod 16, k chunk
    // 4 ks + l / 16 of stage kt.
    const int fr = lane & 15, fq = lane >> 4;
    const int c0 = wn * 16 * half;  // first column of this wave's tiles
    auto aload = [&](int kt, int ks, int i) {
        const unsigned char *sa = lds + (kt & 1) * kStageBytes;
        return *reinterpret_cast<const bf16x8_t *>(
            sa + chunk_at(wm * 64 + 16 * i + fr, 4 * ks + fq));
    };
    auto bload = [&](int kt, int ks, int j) {
        const unsigned char *sb = lds + (kt & 1) * kStageBytes + kPM * kRow;
        return *reinterpret_cast<const bf16x8_t *>(sb + chunk_at(c0 + 16 * j + fr, 4 * ks + fq));
    };
    // A ragged last stage: the A chunks past m hold the next row's elements;
    // zero them in LDS once the stage has landed.
    auto zero_tail = [&](int kt) {
        const int valid = (a.m - kt * kPK) / 8;  // whole chunks still inside m
        unsigned char *sa = lds + (kt & 1) * kStageBytes;
        for (int f = tid; f < kPM * 8; f += kPThreads) {
            const int row = f >> 3, c = f & 7;
            if (c >= valid)
                *reinterpret_cast<u32x4_t *>(sa + chunk_at(row, c)) = u32x4_t{0u, 0u, 0u, 0u};
        }
    };

    // One k-step, column tile by column tile: B fragment j against the 4 A
    // fragments.  The A fragments of the next k-step are read during the
    // first columns, the B fragments RING - 1 columns ahead; the other wave
    // on the SIMD covers what remains of the LDS latency.
    constexpr int RING = NJ % 4 == 0 ? 4 : 3;
    bf16x8_t a0[4], a1[4], br[RING];
    auto kstep = [&](int kt, int ks, bf16x8_t(&acur)[4], bf16x8_t(&anext)[4], bool more) {
        const int nkt = ks ? kt + 1 : kt, nks = ks ^ 1;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if (j + RING - 1 < NJ)
                br[(j + RING - 1) % RING] = bload(kt, ks, j + RING - 1);
            else if (more)
                br[(j + RING - 1) % RING] = bload(nkt, nks, j + RING - 1 - NJ);
            if (more && j < 4)
                anext[j] = aload(nkt, nks, j);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(acur[i], br[j % RING], acc[i][j],
                                                                    0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        if (more && NJ < 4) {
#pragma unroll
            for (int i = NJ; i < 4; ++i)
                anext[i] = aload(nkt, nks, i);
        }
    };

    const bool ragged = a.m % kPK != 0;
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (ragged && nk == 1) {
        zero_tail(0);
        __syncthreads();
    }
    if (nk > 1)
        issue(1, 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
        a0[i] = aload(0, 0, i);
#pragma unroll
    for (int j = 0; j < RING - 1; ++j)
        br[j] = bload(0, 0, j);
    for (int kt = 0; kt < nk; ++kt) {
        // First k-step: its successor is in the same stage.
        kstep(kt, 0, a0, a1, true);
        // Stage kt+1 (issued two k-steps ago) becomes visible before the
        // second k-step prefetches from it.
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (ragged && kt + 2 == nk) {
            zero_tail(kt + 1);
            __syncthreads();
        }
        kstep(kt, 1, a1, a0, kt + 1 < nk);
        // Every wave is done with stage kt's buffer: refill it.
        __syncthreads();
        if (kt + 2 < nk)
            issue(kt + 2, kt & 1);
    }

    // Epilogue, one half of the rows at a time: lane holds C[wm*128 + 16 i +
    // 4 (lane / 16) + e][c0 + 16 j + (lane mod 16)]; round to bf16 into an LDS
    // tile, then write 16-byte row segments.  Wave column 0 stores only its
    // `half` tiles (the instance may be larger); wave column 1's extra tiles
    // lie past the tile's width.
    uint16_t *Cs = reinterpret_cast<uint16_t *>(lds);
    const int nchunk = (width + 7) / 8;
    for (int h = 0; h < 2; ++h) {
        if ((wm >> 1) == h) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    if (wn == 1 || j < half) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            Cs[((wm & 1) * 64 + 16 * i + 4 * fq + e) * kCd + c0 + 16 * j + fr] =
                                to_bf16(acc[i][j][e]);
                    }
        }
        __syncthreads();
        for (int f = tid; f < (kPM / 2) * nchunk; f += kPThreads) {
            const int row = f / nchunk, chunk = f - row * nchunk;
            const int64_t n = n0 + h * (kPM / 2) + row;
            const int j = j0 + 8 * chunk;
            if (n >= a.N)
                continue;
            const u32x4_t v = *reinterpret_cast<const u32x4_t *>(Cs + row * kCd + 8 * chunk);
            if (j + 8 <= a.d && a.ovec) {
                store_stream<uint16_t, 8, true>(a.O + n * a.d + j, v);
            } else if (j >= a.d && j + 8 <= nout && a.kvec) {
                store_stream<uint16_t, 8, true>(a.K + n * a.r + (j - a.d), v);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int c = j + e;
                    const uint16_t x = (uint16_t)(v[e / 2] >> (16 * (e & 1)));
                    if (c >= j0 + width)
                        break;
                    if (c < a.d)
                        a.O[n * a.d + c] = x;
                    else if (c < nout)
                        a.K[n * a.r + (c - a.d)] = x;
                }
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kPThreads, 1) void key_proj_gemm(ProjArgs a)
{
    __shared__ __align__(16) unsigned char lds[2 * kStageBytes];
    // Workgroup b runs on XCD b mod 8; each XCD takes a contiguous range of
    // logical tiles, so the column tiles of one row tile share its L2.
    const int nb = gridDim.x, per = (nb + 7) / 8, xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int full = nb % 8 == 0 ? 8 : nb % 8;  // XCDs that take `per` tiles
    const int t = xcd < full ? xcd * per + slot : full * per + (xcd - full) * (per - 1) + slot;
    const int64_t n0 = (int64_t)(t / a.ncol) * kPM;
    const int c = t % a.ncol;
    const int j0 = c * kPN;
    const int nout = a.d + a.r;
    const int width = c + 1 < a.ncol ? kPN : nout - j0;
    // Wave column 0 covers the first `half` column tiles (of 16), wave
    // column 1 the rest.  All four waves run one instance, of at least `half`
    // tiles (at most 9: 288 columns).
    const int nct = (width + 15) / 16;
    const int half = (nct + 1) / 2;
    if (half <= 4)
        key_proj_tile<4>(a, lds, n0, j0, width, half);
    else if (half <= 8)
        key_proj_tile<8>(a, lds, n0, j0, width, half);
    else
        key_proj_tile<9>(a, lds, n0, j0, width, half);
}

}  // namespace

int check_key_proj_supported(const KeyProjProblem &p, std::string *why)
{
    if (p.dtype != LRAR_DTYPE_BF16) {
        *why = "the key producer runs on bf16 storage (the matrix cores' input type)";
        return LRAR_EUNSUPPORTED;
    }
    if (p.m % 8 != 0) {
        *why = "the key producer needs m % 8 == 0";
        return LRAR_EUNSUPPORTED;
    }
    if (p.m > (1 << 20) || p.d + p.r > (1 << 20)) {
        *why = "the key producer supports m and d + r up to 2^20";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N > ((int64_t)1 << 30)) {
        *why = "N above 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if ((int64_t)key_proj_col_tiles(p.d + p.r) * ((p.N + kPM - 1) / kPM) > INT32_MAX) {
        *why = "too many output tiles for one launch";
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_key_proj(const KeyProjProblem &p, hipStream_t st, std::string *err)
{
    if (p.N == 0)
        return LRAR_OK;
    ProjArgs a;
    a.A = static_cast<const uint16_t *>(p.A);
    a.W = static_cast<const uint16_t *>(p.W);
    a.O = static_cast<uint16_t *>(p.O);
    a.K = static_cast<uint16_t *>(p.K);
    a.N = p.N;
    a.m = (int)p.m;
    a.d = (int)p.d;
    a.r = (int)p.r;
    a.ovec = p.d % 8 == 0 && reinterpret_cast<uintptr_t>(p.O) % 16 == 0;
    a.kvec = p.d % 8 == 0 && p.r % 8 == 0 && reinterpret_cast<uintptr_t>(p.K) % 16 == 0;
    a.ncol = key_proj_col_tiles(p.d + p.r);
    const int64_t tiles = (int64_t)a.ncol * ((p.N + kPM - 1) / kPM);
    hipLaunchKernelGGL(key_proj_gemm, dim3((unsigned)tiles), dim3(kPThreads), 0, st, a);
    return hip_status(hipGetLastError(), "key_proj_gemm launch", err);
}

}  // namespace lrar
