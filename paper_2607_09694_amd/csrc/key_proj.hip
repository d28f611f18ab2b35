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
// layout of a linear layer).  32-wide k-slices (one MFMA k-step) of both go
// straight from memory to LDS with buffer loads (no register staging), in a
// ring of four stages: a slice is issued three k-steps before it is used,
// so its loads have two k-steps of matrix work to land behind, which is
// what the activation streamed from HBM needs.  The buffer resources cover
// only the workgroup's rows, so rows past N or past the output read as
// zero.  LDS rows are 64 bytes with the 16-byte chunks XOR-swizzled by
// (row / 4) mod 4, so that the 16 consecutive rows that one MFMA operand
// read touches fall on distinct banks.  Within a k-step the MFMAs go column
// tile by column tile; the B fragments are read a few columns ahead and the
// next k-step's A fragments during the first columns.
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
constexpr int kPK = 32;              // k per LDS stage (one MFMA k-step)
constexpr int kStages = 4;           // LDS ring
constexpr int kRow = kPK * 2;        // bytes per LDS row of a stage (unpadded)
constexpr int kBlockRows = 1024 / kRow;          // rows per 1 KB block (16)
constexpr int kABlocks = kPM / kBlockRows;       // 1 KB blocks: A part of a stage
constexpr int kBBlocks = kPNMax / kBlockRows;    // ... and W part
constexpr int kStageBytes = (kPM + kPNMax) * kRow;
constexpr int kWaves8 = 8;           // waves per workgroup (2 per SIMD)
constexpr int kLoads = (kABlocks + kBBlocks + kWaves8 - 1) / kWaves8;  // direct loads per wave
// Waves 0 .. kLongWaves-1 issue kLoads loads per stage, the others one fewer.
constexpr int kLongWaves = (kABlocks + kBBlocks) % kWaves8 == 0 ? kWaves8
                                                                 : (kABlocks + kBBlocks) % kWaves8;
constexpr int kCd = kPNMax + 8;      // LDS row stride of the output half-tile (elements)
constexpr int kPThreads = kWaves8 * kWaveSize;
// Buffer resource word 3 for raw (untyped) loads on gfx9-family parts.
constexpr int kRawBufferFlags = 0x00020000;

static_assert(kABlocks % kWaves8 == 0, "A blocks split evenly over the waves");
static_assert(kStages * kStageBytes >= kPM / 2 * kCd * 2, "output half-tile fits the stages");
static_assert(kLoads <= 15, "loads per stage fit the vmcnt immediates below");

// s_waitcnt immediate (gfx9 encoding): at most n vector-memory operations
// outstanding; expcnt and lgkmcnt left at their maxima (not waited on).
constexpr int vmcnt_at_most(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

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

// LDS placement of 16-byte chunk c (0..3) of stage row `row`: rows are 64
// bytes, and the chunk is XOR-swizzled with (row / 4) mod 4, so the 16
// consecutive rows that one MFMA operand read touches spread over all banks.
__device__ __forceinline__ int chunk_at(int row, int c) { return row * kRow + 16 * (c ^ ((row >> 2) & 3)); }

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
    // wave's u-th load fills 1 KB block blk = wave + 8 u, 16 rows of 64
    // bytes: lane l writes bytes 16 l .. 16 l + 15 of the block, i.e. block
    // row l / 4, placed chunk l mod 4, which holds global chunk
    // (l mod 4) ^ swizzle.  Blocks 0 .. kABlocks-1 are A's rows, the rest
    // W's.  The swizzle (row / 4) mod 4 of block row l / 4 is (l / 16) mod 4
    // for every block, so each lane needs one offset; the block's first row
    // and the k offset are scalar.  The buffer resources cover the
    // workgroup's rows of A and of W only, so rows past N, past the tile or
    // past d + r read as zero.  A chunk past m reads the next row's first
    // elements; it is zeroed in LDS (zero_tail).
    const int voff = (lane >> 2) * a.m * 2 + 16 * ((lane & 3) ^ ((lane >> 4) & 3));
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
                                                         voff, blk * kBlockRows * a.m * 2 + kbytes,
                                                         0, 0);
            else if (blk < kABlocks + kBBlocks)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    bres, (lds_void_t *)(sb + 1024 * blk), 16, voff,
                    (blk - kABlocks) * kBlockRows * a.m * 2 + kbytes, 0, 0);
        }
    };

    f32x4_t acc[4][NJ];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // Operand fragments: lane l reads row base + l mod 16, k chunk l / 16
    // of stage kt.
    const int fr = lane & 15, fq = lane >> 4;
    const int c0 = wn * 16 * half;  // first column of this wave's tiles
    // sbase: byte offset of the stage's buffer, recomputed (not hoisted) at
    // every k-step so that one address register serves each of the ring's
    // four buffers.
    const int aoff = chunk_at(wm * 64 + fr, fq), boff = kPM * kRow + chunk_at(c0 + fr, fq);
    auto stage_base = [&](int kt) {
        int sbase = (kt % kStages) * kStageBytes;
        asm volatile("" : "+s"(sbase));
        return sbase;
    };
    auto aload = [&](int sbase, int i) {
        return *reinterpret_cast<const bf16x8_t *>(lds + sbase + aoff + 16 * kRow * i);
    };
    auto bload = [&](int sbase, int j) {
        return *reinterpret_cast<const bf16x8_t *>(lds + sbase + boff + 16 * kRow * j);
    };
    // A ragged last stage: the A chunks past m hold the next row's elements;
    // zero them in LDS once the stage has landed.
    auto zero_tail = [&](int kt) {
        const int valid = (a.m - kt * kPK) / 8;  // whole chunks still inside m
        unsigned char *sa = lds + (kt % kStages) * kStageBytes;
        for (int f = tid; f < kPM * 4; f += kPThreads) {
            const int row = f >> 2, c = f & 3;
            if (c >= valid)
                *reinterpret_cast<u32x4_t *>(sa + chunk_at(row, c)) = u32x4_t{0u, 0u, 0u, 0u};
        }
    };
    // Wait until at most the last `ahead` stages issued by this wave are
    // still in flight (waves 0 .. kLongWaves-1 issue one load more).
    auto wait_stages = [&](int ahead) {
        if (ahead == 0)
            __builtin_amdgcn_s_waitcnt(vmcnt_at_most(0));
        else if (wave < kLongWaves)
            __builtin_amdgcn_s_waitcnt(vmcnt_at_most(kLoads));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_at_most(kLoads - 1));
    };

    // One k-step, column tile by column tile: B fragment j against the 4 A
    // fragments.  The A fragments of the next k-step are read during the
    // first columns, the B fragments RING - 1 columns ahead; the other wave
    // on the SIMD covers what remains of the LDS latency.
    constexpr int RING = NJ % 4 == 0 ? 4 : 3;
    bf16x8_t a0[4], a1[4], br[RING];
    auto kstep = [&](int kt, bf16x8_t(&acur)[4], bf16x8_t(&anext)[4], bool more) {
        const int scur = stage_base(kt), snext = stage_base(kt + 1);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if (j + RING - 1 < NJ)
                br[(j + RING - 1) % RING] = bload(scur, j + RING - 1);
            else if (more)
                br[(j + RING - 1) % RING] = bload(snext, j + RING - 1 - NJ);
            if (more && j < 4)
                anext[j] = aload(snext, j);
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
                anext[i] = aload(snext, i);
        }
    };

    // The ring: before k-step kt runs, stages kt and kt + 1 have landed and
    // are visible, stage kt + 2 is in flight and stage kt + 3 is issued into
    // the buffer that k-step kt - 1 has just released.  The barrier at the
    // end of k-step kt makes stage kt + 2 visible (k-step kt reads its
    // successor's first fragments) and releases stage kt's buffer.  The
    // barriers order LDS only, so the stages issued ahead stay in flight.
    const bool ragged = a.m % kPK != 0;
    for (int s = 0; s < kStages - 1 && s < nk; ++s)
        issue(s, s);
    // Stages 0 and 1 visible; stage 2 may stay in flight.
    wait_stages(nk > 2 ? 1 : 0);
    lds_barrier();
    if (ragged && nk <= 2) {
        zero_tail(nk - 1);
        lds_barrier();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
        a0[i] = aload(0, i);
#pragma unroll
    for (int j = 0; j < RING - 1; ++j)
        br[j] = bload(0, j);
    // Main loop: two k-steps per trip (so the A fragment registers
    // alternate), each with a successor, so every prefetch is unconditional.
    int kt = 0;
    for (; kt + 2 < nk; kt += 2) {
        if (kt + 3 < nk)
            issue(kt + 3, (kt + 3) % kStages);
        kstep(kt, a0, a1, true);
        wait_stages(kt + 3 < nk ? 1 : 0);
        lds_barrier();
        if (ragged && kt + 3 == nk) {
            zero_tail(kt + 2);
            lds_barrier();
        }
        if (kt + 4 < nk)
            issue(kt + 4, (kt + 4) % kStages);
        kstep(kt + 1, a1, a0, true);
        wait_stages(kt + 4 < nk ? 1 : 0);
        lds_barrier();
        if (ragged && kt + 4 == nk) {
            zero_tail(kt + 3);
            lds_barrier();
        }
    }
    // The last one or two k-steps: every stage has landed, is visible and,
    // if ragged, zeroed; nothing more is written to LDS before the epilogue.
    kstep(kt, a0, a1, kt + 1 < nk);
    if (kt + 1 < nk)
        kstep(kt + 1, a1, a0, false);
    lds_barrier();

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
    __shared__ __align__(16) unsigned char lds[kStages * kStageBytes];
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
