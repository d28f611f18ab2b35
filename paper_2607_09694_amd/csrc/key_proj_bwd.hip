// Backward of the projected-key producer (Sec. 3.3, Eq. fused_projection).
// The forward is one linear map C = A W^T with C = [O, K] (the d value
// columns, then the r key columns).  For upstream gradients G = [dO, dK]
// ([N][d + r], split at column d like C) the chain rule gives two GEMMs:
//     dA[N][m]     = G W            (reduction over the d + r outputs)
//     dW[d + r][m] = G^T A          (reduction over the N tokens)
// so the key rows of W cost r more reduction steps in dA and r more rows of
// dW, the same r / d overhead as in the forward.
//
// One tile kernel serves both.  A workgroup of 4 waves computes a 128 x 128
// output tile with v_mfma_f32_16x16x32_bf16 and fp32 accumulators (each
// wave a 64 x 64 quarter, 16 MFMA tiles).  The reduction runs in stages of
// 64: every stage is loaded from memory into registers while the previous
// one feeds the MFMAs, then written to LDS.  An MFMA operand fragment holds,
// per lane, 8 consecutive reduction steps of one output index.  Of the four
// operand reads only G in dA has the reduction index contiguous in memory
// (its LDS rows are output indices, read 16 bytes a lane); W in dA and both
// G and A in dW have the output index contiguous instead.  Those
// stay in that layout in LDS (rows are reduction steps, 16-byte chunks
// copied as loaded) and are transposed by the read: gfx950's ds_read_b64_tr_b16
// gives lane i of a 16-lane group element i mod 4 of the 8 bytes addressed
// by lane i / 4 + 4 e, for e = 0..3.  Pointing lane s of the group at
// reduction step s / 4 and output indices 4 (s mod 4) .. +3 therefore hands
// lane i four consecutive reduction steps of output index i; two such reads
// make an MFMA operand fragment.  Rows of the reduction-contiguous operand
// are padded to 72 elements and rows of a transposed one to 144, which
// spreads one operand read over the banks.
//
// dA rounds to bf16 (nearest even).  dW is written in fp32, so that a caller
// can add it to fp32 master gradients without a second rounding; its token
// reduction is split over P workgroups per tile when the tile grid alone
// would not fill the chip, each writing an fp32 partial into the caller's
// workspace, and a second kernel sums the partials in split order.  Every
// sum has a fixed order, so the results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <string>

#include "route_common.h"

namespace lrar {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kBM = 128;                          // output rows per tile
constexpr int kBN = 128;                          // output columns per tile
constexpr int kBK = 64;                           // reduction steps per stage
constexpr int kLd = kBK + 8;                      // LDS row stride (elements)
constexpr int kBThreads = 256;                    // 4 waves
constexpr int kRowChunks = kBM * kBK / 8 / kBThreads;       // 4: k-contiguous loads per lane
constexpr int kTs = kBN + 16;                     // LDS row stride of a transposed operand
constexpr int kTChunks = kBK * kBN / 8 / kBThreads;         // 4: transposed-operand loads per lane
constexpr int kSlots = 2 * 256;                   // workgroups resident at once (2 per CU)

static_assert(kRowChunks == 4 && kTChunks == 4, "stage loads split evenly over the lanes");
constexpr int kCs = kBN + 8;                      // LDS row stride of the staged bf16 dA tile
constexpr int kCf = kBN + 4;                      // ... of a staged fp32 dW half-tile (floats)
static_assert(kBK * kTs == kBM * kLd, "both LDS layouts of an operand take the same space");
static_assert(kBM * kCs <= 2 * kBM * kLd && (kBM / 2) * kCf * 2 <= 2 * kBM * kLd,
              "the staged output fits the operand stages");

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef __attribute__((address_space(3))) char lds_char_t;

struct BwdArgs {
    const uint16_t *A;   // [N][m]
    const uint16_t *W;   // [d + r][m]
    const uint16_t *dO;  // [N][d] or NULL (d = 0)
    const uint16_t *dK;  // [N][r] or NULL (r = 0)
    uint16_t *dA;        // [N][m]
    float *dst;          // dW [d + r][m] (one split) or partials [P][d + r][m]
    int64_t N;
    int64_t per;         // tokens per split (a multiple of kBK)
    int m, d, r;
    int ntn;             // column tiles
};

__device__ __forceinline__ u32x4_t zero4() { return u32x4_t{0u, 0u, 0u, 0u}; }

// 8 consecutive outputs o .. o+7 of token n from [dO, dK] (o % 8 == 0, and
// d % 8 == 0, so the 8 never straddle the split).
__device__ __forceinline__ u32x4_t g_chunk(const BwdArgs &a, int64_t n, int o)
{
    if (o < a.d)
        return *reinterpret_cast<const u32x4_t *>(a.dO + n * a.d + o);
    return *reinterpret_cast<const u32x4_t *>(a.dK + n * a.r + (o - a.d));
}

// MFMA operand fragment from a transposed operand in LDS (row = reduction
// step, kTs elements per row): lane l receives reduction steps 32 ks +
// 8 (l / 16) .. +7 of output index base + l mod 16.  Within each 16-lane
// group, lane s addresses step s / 4 (then s / 4 + 4) and output indices
// base + 4 (s mod 4) .. +3; the transposing read regroups the elements.
__device__ __forceinline__ bf16x8_t frag_tr(const uint16_t *S, int ks, int base, int lane)
{
    const int row = 32 * ks + 8 * (lane >> 4) + ((lane & 15) >> 2);
    const int col = base + 4 * (lane & 3);
    lds_char_t *p = (lds_char_t *)(S) + 2 * (row * kTs + col);
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)p);
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(p + 2 * 4 * kTs));
    return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// DW = false: C = dA tile (rows: tokens, columns: input features, reduction:
//             the d + r outputs).  X = G rows (k-contiguous), Y = W (transposed).
// DW = true:  C = dW tile (rows: outputs, columns: input features, reduction:
//             the tokens of split blockIdx.y).  X = G (transposed), Y = A
//             (transposed).
template <bool DW>
__global__ __launch_bounds__(kBThreads) void key_proj_bwd_gemm(BwdArgs a)
{
    __shared__ __align__(16) uint16_t lds[2 * kBM * kLd];
    uint16_t *const Xs = lds;
    uint16_t *const Ys = lds + kBM * kLd;

    const int tid = threadIdx.x;
    const int lane = tid % kWaveSize, wave = tid / kWaveSize;
    const int wm = wave >> 1, wn = wave & 1;
    const int nout = a.d + a.r;
    const int64_t tm = blockIdx.x / a.ntn;
    const int tn = blockIdx.x % a.ntn;
    const int64_t row0 = tm * kBM;  // token (dA) or output (dW)
    const int col0 = tn * kBN;      // input feature
    const int64_t rows = DW ? nout : a.N;
    const int64_t kbeg = DW ? (int64_t)blockIdx.y * a.per : 0;
    const int64_t kend = DW ? min(a.N, kbeg + a.per) : nout;
    const int nk = (int)((kend - kbeg + kBK - 1) / kBK);

    // Stage registers: 4 chunks of 8 elements per operand.  A transposed
    // operand's chunk u is reduction step q / 16 of the stage, output indices
    // 8 (q mod 16) .. +7 of the tile, with q = tid + 256 u.
    u32x4_t xr[4], yr[4];
    auto fetch = [&](int kt) {
        const int64_t k0 = kbeg + (int64_t)kt * kBK;
        if (!DW) {
#pragma unroll
            for (int u = 0; u < kRowChunks; ++u) {
                const int q = tid + kBThreads * u, row = q >> 3, kc = q & 7;
                const int64_t n = row0 + row;
                const int64_t o = k0 + 8 * kc;
                xr[u] = (n < a.N && o < kend) ? g_chunk(a, n, (int)o) : zero4();
            }
        }
        const uint16_t *Y = DW ? a.A : a.W;
#pragma unroll
        for (int u = 0; u < kTChunks; ++u) {
            const int q = tid + kBThreads * u, ks = q >> 4, mc = q & 15;
            const int64_t k = k0 + ks;
            if (DW) {
                const int64_t o = row0 + 8 * mc;
                xr[u] = (o < nout && k < kend) ? g_chunk(a, k, (int)o) : zero4();
            }
            const int j = col0 + 8 * mc;
            yr[u] = (j < a.m && k < kend)
                        ? *reinterpret_cast<const u32x4_t *>(Y + k * a.m + j) : zero4();
        }
    };
    auto put_tr = [&](uint16_t *S, const u32x4_t *v) {
#pragma unroll
        for (int u = 0; u < kTChunks; ++u) {
            const int q = tid + kBThreads * u, ks = q >> 4, mc = q & 15;
            *reinterpret_cast<u32x4_t *>(S + ks * kTs + 8 * mc) = v[u];
        }
    };
    auto put = [&]() {
        if (!DW) {
#pragma unroll
            for (int u = 0; u < kRowChunks; ++u) {
                const int q = tid + kBThreads * u, row = q >> 3, kc = q & 7;
                *reinterpret_cast<u32x4_t *>(Xs + row * kLd + 8 * kc) = xr[u];
            }
        } else {
            put_tr(Xs, xr);
        }
        put_tr(Ys, yr);
    };

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // Operand fragments: lane l reads row 16 i + l mod 16 of its quarter,
    // elements 32 ks + 8 (l / 16) .. +7 of the stage.
    const int fr = lane & 15, fq = lane >> 4;
    if (nk > 0) {
        fetch(0);
        put();
        __syncthreads();
    }
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk)
            fetch(kt + 1);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8_t xf[4], yf[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                xf[i] = DW ? frag_tr(Xs, ks, wm * 64 + 16 * i, lane)
                           : *reinterpret_cast<const bf16x8_t *>(
                                 Xs + (wm * 64 + 16 * i + fr) * kLd + 32 * ks + 8 * fq);
                yf[i] = frag_tr(Ys, ks, wn * 64 + 16 * i, lane);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf[i], yf[j], acc[i][j],
                                                                        0, 0, 0);
        }
        __syncthreads();
        if (kt + 1 < nk) {
            put();
            __syncthreads();
        }
    }

    // Epilogue (every wave is past its last LDS read): lane holds
    // C[16 i + 4 (l / 16) + e][16 j + l mod 16] of its quarter.  The tile is
    // staged through LDS and written as 16-byte row segments: dA whole, as
    // bf16; dW in two halves of 64 rows, as fp32.
    if (!DW) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    lds[(wm * 64 + 16 * i + 4 * fq + e) * kCs + wn * 64 + 16 * j + fr] =
                        to_bf16(acc[i][j][e]);
        __syncthreads();
        for (int f = tid; f < kBM * (kBN / 8); f += kBThreads) {
            const int row = f >> 4, ch = f & 15;
            const int64_t n = row0 + row;
            const int c = col0 + 8 * ch;
            if (n < rows && c < a.m)
                *reinterpret_cast<u32x4_t *>(a.dA + n * a.m + c) =
                    *reinterpret_cast<const u32x4_t *>(lds + row * kCs + 8 * ch);
        }
    } else {
        float *const Cf = reinterpret_cast<float *>(lds);
        float *const dst = a.dst + (int64_t)blockIdx.y * nout * a.m;
        for (int h = 0; h < 2; ++h) {
            if (wm == h) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            Cf[(16 * i + 4 * fq + e) * kCf + wn * 64 + 16 * j + fr] = acc[i][j][e];
            }
            __syncthreads();
            for (int f = tid; f < (kBM / 2) * (kBN / 4); f += kBThreads) {
                const int row = f >> 5, ch = f & 31;
                const int64_t o = row0 + (kBM / 2) * h + row;
                const int c = col0 + 4 * ch;
                if (o < rows && c < a.m)
                    *reinterpret_cast<f32x4_t *>(dst + o * a.m + c) =
                        *reinterpret_cast<const f32x4_t *>(Cf + row * kCf + 4 * ch);
            }
            __syncthreads();
        }
    }
}

// dW[x] = sum over the P partials in split order (P = 0 writes zeros: the
// gradient of W over no tokens).
__global__ __launch_bounds__(kBThreads) void key_proj_bwd_reduce(const float *part, float *dW,
                                                               int64_t count4, int P)
{
    const int64_t stride = (int64_t)gridDim.x * kBThreads;
    const int64_t plane = count4 * 4;
    for (int64_t x = (int64_t)blockIdx.x * kBThreads + threadIdx.x; x < count4; x += stride) {
        f32x4_t s = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        for (int p = 0; p < P; ++p)
            s += *reinterpret_cast<const f32x4_t *>(part + p * plane + 4 * x);
        *reinterpret_cast<f32x4_t *>(dW + 4 * x) = s;
    }
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

// Token splits of dW: as many as let every workgroup of the launch be
// resident at once (a second, partial round of workgroups would cost a
// whole round's time), each split a multiple of one stage.  P = 0 when there
// are no tokens.
void key_proj_bwd_splits(int64_t N, int64_t m, int64_t nout, int64_t *P, int64_t *per)
{
    if (N == 0) {
        *P = 0;
        *per = kBK;
        return;
    }
    const int64_t tiles = ceil_div(nout, kBM) * ceil_div(m, kBN);
    const int64_t want = std::max((int64_t)1, std::min(kSlots / tiles, ceil_div(N, kBK)));
    *per = ceil_div(ceil_div(N, want), kBK) * kBK;
    *P = ceil_div(N, *per);
}

size_t key_proj_bwd_workspace_bytes(int64_t N, int64_t m, int64_t d, int64_t r)
{
    int64_t P, per;
    key_proj_bwd_splits(N, m, d + r, &P, &per);
    return P > 1 ? (size_t)P * (size_t)(d + r) * (size_t)m * sizeof(float) : 0;
}

int check_key_proj_bwd_supported(const KeyProjProblem &p, std::string *why)
{
    if (p.dtype != LRAR_DTYPE_BF16) {
        *why = "the key producer's backward runs on bf16 storage (the matrix cores' input type)";
        return LRAR_EUNSUPPORTED;
    }
    if (p.m % 8 != 0 || p.d % 8 != 0 || p.r % 8 != 0) {
        *why = "the key producer's backward needs m, d and r multiples of 8";
        return LRAR_EUNSUPPORTED;
    }
    if (p.m > (1 << 20) || p.d + p.r > (1 << 20)) {
        *why = "the key producer's backward supports m and d + r up to 2^20";
        return LRAR_EUNSUPPORTED;
    }
    if (p.N > ((int64_t)1 << 30)) {
        *why = "N above 2^30 tokens";
        return LRAR_EUNSUPPORTED;
    }
    if (ceil_div(p.N, kBM) * ceil_div(p.m, kBN) > INT32_MAX) {
        *why = "too many output tiles for one launch";
        return LRAR_EUNSUPPORTED;
    }
    return LRAR_OK;
}

int launch_key_proj_bwd(const KeyProjProblem &p, const void *dO, const void *dK, void *dA,
                        float *dW, void *workspace, hipStream_t st, std::string *err)
{
    BwdArgs a;
    a.A = static_cast<const uint16_t *>(p.A);
    a.W = static_cast<const uint16_t *>(p.W);
    a.dO = static_cast<const uint16_t *>(dO);
    a.dK = static_cast<const uint16_t *>(dK);
    a.dA = static_cast<uint16_t *>(dA);
    a.N = p.N;
    a.m = (int)p.m;
    a.d = (int)p.d;
    a.r = (int)p.r;
    a.ntn = (int)ceil_div(p.m, kBN);
    const int64_t nout = p.d + p.r;
    int64_t P;
    key_proj_bwd_splits(p.N, p.m, nout, &P, &a.per);
    if (p.N > 0) {
        const int64_t tiles = ceil_div(p.N, kBM) * a.ntn;
        hipLaunchKernelGGL(key_proj_bwd_gemm<false>, dim3((unsigned)tiles), dim3(kBThreads), 0,
                           st, a);
        int rc = hip_status(hipGetLastError(), "key_proj_bwd_gemm (dA) launch", err);
        if (rc)
            return rc;
        a.dst = P > 1 ? static_cast<float *>(workspace) : dW;
        hipLaunchKernelGGL(key_proj_bwd_gemm<true>,
                           dim3((unsigned)(ceil_div(nout, kBM) * a.ntn), (unsigned)P),
                           dim3(kBThreads), 0, st, a);
        if ((rc = hip_status(hipGetLastError(), "key_proj_bwd_gemm (dW) launch", err)))
            return rc;
    }
    if (P != 1) {
        const int64_t count4 = nout * p.m / 4;
        const int64_t groups = std::max((int64_t)1, std::min(ceil_div(count4, kBThreads), (int64_t)4096));
        hipLaunchKernelGGL(key_proj_bwd_reduce, dim3((unsigned)groups), dim3(kBThreads), 0, st,
                           static_cast<const float *>(workspace), dW, count4, (int)P);
        return hip_status(hipGetLastError(), "key_proj_bwd_reduce launch", err);
    }
    return LRAR_OK;
}

}  // namespace lrar
