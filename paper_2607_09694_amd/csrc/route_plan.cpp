// Launch plans of the routing kernels: which kernel instance, grid and LDS
// size serve a validated problem, and the limits beyond which none does.
// Host code only.
#include "route_common.h"

namespace lrar {

namespace {

constexpr int kMaxSourcesFwd = 1024;
constexpr int kMaxSourcesBwd = 512;
constexpr int kMaxRankBwd = 256;

// Token counts up to which the forward splits each token's sources over the
// four waves of a workgroup (measured on MI355X at 49 sources, d = 1024: the
// split is ahead up to these counts, level with or behind one wave per token
// above them).  LRAR_WG_SPLIT_MAX_TOKENS overrides both.
#ifdef LRAR_WG_SPLIT_MAX_TOKENS
constexpr int64_t kWgSplitLowRank = LRAR_WG_SPLIT_MAX_TOKENS;
constexpr int64_t kWgSplitFull = LRAR_WG_SPLIT_MAX_TOKENS;
#else
constexpr int64_t kWgSplitLowRank = 2048;
constexpr int64_t kWgSplitFull = 1024;
#endif

int round_up(int x, int m) { return (x + m - 1) / m * m; }

}  // namespace

void plan_wg_split(const Problem &p, Plan *pl)
{
    if (p.N > (p.mode == LRAR_MODE_FULL ? kWgSplitFull : kWgSplitLowRank) || p.S < 2)
        return;
    pl->wg_split = true;
    pl->nblocks = (int)p.N;
    const size_t row = (size_t)pl->nch * kWaveSize * pl->vec;
    // Scores in LDS (low-rank keys only), per-wave statistics, the
    // accumulators of waves 1..kWaves-1.
    pl->s_pad = round_up((int)((p.S + kWaves - 1) / kWaves), 4);
    const size_t scores = p.mode == LRAR_MODE_FULL ? 0 : (size_t)kWaves * pl->s_pad;
    pl->lds = (scores + 2 * kWaves + (kWaves - 1) * row) * sizeof(float);
}

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
        // holds its online-softmax state in registers.  (The plan is that of
        // one token per wave; route_fwd_lr's launch scales it to its TW.)
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


int hip_status(hipError_t e, const char *what, std::string *err)
{
    if (e == hipSuccess)
        return LRAR_OK;
    *err = std::string(what) + ": " + hipGetErrorString(e);
    return LRAR_EHIP;
}


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

}  // namespace lrar
