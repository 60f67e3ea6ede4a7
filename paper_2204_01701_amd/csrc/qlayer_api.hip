// qlayer_api.hip -- host side of the C ABI declared in include/qlayer.h:
// argument validation, tile-configuration and split-K planning, workspace
// carving and kernel launches on the caller's stream.  Nothing here touches
// tensor data on the host and nothing allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <mutex>

#include "qlayer.h"
#include "qconv_aux.h"
#include "qconv_bwd_data.h"
#include "qconv_bwd_data_wide.h"
#include "qconv_bwd_weight.h"
#include "qconv_depthwise.h"
#include "qconv_fwd.h"
#include "qconv_fwd_smallc.h"
#include "qconv_generic.h"

namespace ql {
// The 16 zero bytes masked-off lanes of the pipelined kernels load.
__device__ __attribute__((aligned(16))) uint32_t g_zero16[4] = {0u, 0u, 0u, 0u};
}  // namespace ql

namespace {
// Device address of g_zero16 on the current device, resolved once per device
// (std::call_once: host threads calling concurrently see one resolution).
constexpr int kMaxDevices = 64;
const void *zero_page() {
    static std::once_flag once[kMaxDevices];
    static const void *addr[kMaxDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::call_once(once[dev], [dev] {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(ql::g_zero16)) == hipSuccess) addr[dev] = p;
    });
    return addr[dev];
}
}  // namespace

using namespace ql;

namespace {

constexpr int kNumCUs = 256;         // MI355X compute units
constexpr size_t kAlign = 256;
constexpr long long kMaxElems = (1LL << 31) - 1;  // 32-bit element offsets in the kernels
constexpr size_t kMaxSplitBytes = 128ull << 20;  // cap on split-K partial sums (written + read once)
// Split-K cost model, in units of one K step of one workgroup alone on a CU:
// a CU holding two co-resident workgroups finishes both in kSharedRound steps
// per step each (the second one hides the first one's latency), and one unit
// of time moves about kBytesPerStep bytes of partial sums through HBM.
constexpr double kSharedRound = 1.25;
constexpr double kBytesPerStep = 3.2e6;
constexpr double kReduceSteps = 6.0;  // the reduction kernel's launch and ramp

// Tuning override: QLAYER_<NAME>=<int> replaces a planner choice (for sweeps).
int env_override(const char *name, int dflt) {
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    return std::atoi(v);
}

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

struct Geom {
    int N, C, H, W, O, KH, KW, SH, SW, PH, PW, HO, WO;
    ql_dtype dt;
    int ne;  // neuron type (NEURON_*)
    bool dw; // depthwise (groups == C == O)
    int om() const { return om_of_neuron(ne); }
    int terms() const { return om_terms(om()); }
    size_t esize() const { return dt == QL_BF16 ? 2 : 4; }
    int vec() const { return dt == QL_BF16 ? 8 : 4; }
    // Few input channels that are not a multiple of the 16-byte vector (e.g.
    // 3-channel images): X and W_t are copied zero-padded to cpad() channels.
    bool pad_small_c() const { return C % vec() != 0 && C < 2 * vec(); }
    int cpad() const { return (C + vec() - 1) / vec() * vec(); }
};

ql_status make_geom(const ql_conv_desc *d, Geom &g) {
    if (!d) return QL_EINVAL;
    if (d->n <= 0 || d->c <= 0 || d->h <= 0 || d->w <= 0 || d->o <= 0 || d->kh <= 0 || d->kw <= 0)
        return QL_EINVAL;
    if (d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0) return QL_EINVAL;
    if (d->dtype != QL_F32 && d->dtype != QL_BF16) return QL_EINVAL;
    if ((int)d->neuron < NEURON_QUADRA || (int)d->neuron > NEURON_T2) return QL_EINVAL;
    const long long eh = (long long)d->h + 2LL * d->pad_h - d->kh;
    const long long ew = (long long)d->w + 2LL * d->pad_w - d->kw;
    if (eh < 0 || ew < 0) return QL_EINVAL;  // empty output
    g.N = d->n; g.C = d->c; g.H = d->h; g.W = d->w; g.O = d->o; g.KH = d->kh; g.KW = d->kw;
    g.SH = d->stride_h; g.SW = d->stride_w; g.PH = d->pad_h; g.PW = d->pad_w;
    g.HO = (int)(eh / d->stride_h + 1);
    g.WO = (int)(ew / d->stride_w + 1);
    g.dt = d->dtype;
    g.ne = (int)d->neuron;
    if (d->groups != 0 && d->groups != 1 && d->groups != d->c) return QL_EUNSUPPORTED;
    g.dw = d->groups == d->c && d->c > 1;
    if (g.dw && d->o != d->c) return QL_EINVAL;  // one output channel per group
    if (g.dw && 3LL * d->kh * d->kw * kDwCB * 4 > 64 * 1024) return QL_EUNSUPPORTED;  // filters staged in LDS
    // the shortcut of T4 + identity adds input channel o at the same pixel
    if (g.ne == NEURON_T4I && (g.C != g.O || g.HO != g.H || g.WO != g.W)) return QL_EINVAL;
    const long long nx = (long long)g.N * g.H * g.W * g.C;
    const long long ny = (long long)g.N * g.HO * g.WO * g.O;
    const long long nw = (long long)g.O * g.KH * g.KW * g.C;
    if (nx > kMaxElems || ny > kMaxElems || 3 * nw > kMaxElems || g.H + 2LL * g.PH > kMaxElems ||
        g.W + 2LL * g.PW > kMaxElems)
        return QL_EUNSUPPORTED;
    return QL_OK;
}

ql_status linear_geom(const ql_linear_desc *d, Geom &g) {
    if (!d) return QL_EINVAL;
    ql_conv_desc c{d->batch, d->in, 1, 1, d->out, 1, 1, 1, 1, 0, 0, d->dtype, d->neuron, 1};
    return make_geom(&c, g);
}

// Split-K planning.  The workgroups run in rounds of kNumCUs * slots (slots =
// workgroups one CU can hold at once); the split count minimises the modelled
// time: K steps per split times the rounds' cost, plus the traffic of the
// partial sums and the reduction.  A count that leaves a few CUs with a second
// workgroup in the last round costs a whole shared round, which the search
// avoids.  At least min_stages K steps per split, at most kMaxSplitBytes of
// partial sums (bytes_per_split each).
void plan_splits(int tiles, int stages_total, int min_stages, size_t bytes_per_split, int slots, int &splits,
                 int &sps) {
    const int cap_bytes = (int)std::max<size_t>(1, kMaxSplitBytes / std::max<size_t>(bytes_per_split, 1));
    const int s_max = std::max(1, std::min(stages_total / std::max(min_stages, 1), cap_bytes));
    double best = 0.0;
    splits = 1;
    for (int s = 1; s <= s_max; ++s) {
        const int per = cdiv(stages_total, s);
        const int eff = cdiv(stages_total, per);
        if (eff != s) continue;  // the same partition as a smaller count
        const long long wgs = (long long)tiles * eff;
        const long long round = (long long)kNumCUs * std::max(slots, 1);
        const long long full = wgs / round, rest = wgs % round;
        double rounds = (double)full * (slots > 1 ? kSharedRound : 1.0);
        if (rest > 0) rounds += rest > kNumCUs ? kSharedRound : 1.0;
        double t = per * rounds;
        if (eff > 1) t += (double)eff * bytes_per_split * 2.0 / kBytesPerStep + kReduceSteps;
        if (s == 1 || t < best) {
            best = t;
            splits = eff;
        }
    }
    sps = cdiv(stages_total, splits);
    splits = cdiv(stages_total, sps);
}

// Taps (r, q) in bounds for output position pos = (oh, ow): a bit mask.
uint32_t tap_mask(const Geom &g, int pos) {
    const int oh = pos / g.WO, ow = pos % g.WO;
    const int h0 = oh * g.SH - g.PH, w0 = ow * g.SW - g.PW;
    uint32_t m = 0;
    for (int r = 0; r < g.KH; ++r)
        for (int q = 0; q < g.KW; ++q)
            if (h0 + r >= 0 && h0 + r < g.H && w0 + q >= 0 && w0 + q < g.W) m |= 1u << (r * g.KW + q);
    return m;
}

// Position-major pixel order (column m = position m / N of image m % N): the
// most in-bounds taps of any pixel tile of `bcol` columns (the union over
// the positions it spans).
int pm_max_taps(const Geom &g, int bcol, long long M) {
    int best = 0;
    for (long long m0 = 0; m0 < M; m0 += bcol) {
        const long long m1 = std::min(M, m0 + bcol) - 1;
        uint32_t u = 0;
        for (long long pos = m0 / g.N; pos <= m1 / g.N; ++pos) u |= tap_mask(g, (int)pos);
        best = std::max(best, __builtin_popcount(u));
    }
    return best;
}

// Whether to use the position-major order: forced by `env` (0 / 1), else on
// padded maps of at most 4 positions (2 x 2 maps of a 3 x 3 filter: every
// position has 4 taps in bounds).  Measured on larger maps (4 x 4, 8 x 8),
// the order is slower: the interior positions keep every tap, so their tiles
// bound the kernel's time, and a tile of one position no longer re-reads the
// X rows its neighbouring pixels share across taps from the caches.
bool pm_default(const Geom &g, int env) {
    if (env >= 0) return env != 0;
    return g.HO * g.WO <= 4 && (g.PH > 0 || g.PW > 0);
}

// ---------------------------------------------------------------------------
// Forward planning.
// ---------------------------------------------------------------------------
// Pipelined forward tile configurations (rows = output channels per term,
// columns = output pixels; per-wave tile in parentheses; 4 waves unless noted):
//   0: 128 x 128 (32 x 128), 1: 64 x 256 (32 x 128), 2: 128 x 128 (64 x 64), 3: 64 x 128 (32 x 64),
//   4: 128 x 256 (32 x 128, 8 waves), 5: 128 x 256 (64 x 64, 8 waves).
// Larger workgroup tiles move fewer bytes through the vector-memory address
// path per MFMA: 32768 (1/BCOL + 1/(3 BR)) bytes.
constexpr int kFwdCfgs = 6;
constexpr int kFwdBR[kFwdCfgs] = {128, 64, 128, 64, 128, 128};
constexpr int kFwdBCOL[kFwdCfgs] = {128, 256, 128, 128, 256, 256};
// Workgroups one CU holds at once (limited by LDS stages and registers).
constexpr int kFwdSlots[kFwdCfgs] = {1, 1, 1, 2, 1, 1};

struct FwdPlan {
    int cfg;  // pipelined: index into kFwd*; generic: 0: 128 x 128, 1: 64 x 128
    int BR, BCOL, KE, slots;
    int row_tiles, col_tiles, splits, sps, stages_total;
    bool veck;
    bool smallc;  // KH KW C + bias columns <= 32, 32 or 64 output channels: qconv_fwd_smallc_kernel, no workspace
    bool ca;  // channel-aligned K steps (C a multiple of KE, at most 32 taps): every step within one tap
    bool pm;  // position-major pixel order, K steps of padding-only taps skipped (FwdArgs)
    bool pad;                      // X and W_t zero-padded to Cp channels first
    int Cp;
    size_t xpad_bytes, wpad_bytes;  // workspace: [X padded][W_a, W_b, W_c padded][split partials][X o X]
    size_t part_bytes;
    size_t xsq_bytes;               // T2 with 16-byte channel vectors: X o X formed once by a pre-pass
    size_t ws_bytes;
};

FwdPlan plan_fwd(const Geom &g) {
    FwdPlan p{};
    const int bias_cols = g.dt == QL_BF16 ? smallc_bias_cols<uint16_t>() : smallc_bias_cols<float>();
    if (g.ne == NEURON_QUADRA && g.C * g.KH * g.KW + bias_cols <= kSmallcK && (g.O == 32 || g.O == 64) &&
        env_override("QLAYER_FWD_SMALLC", 1) != 0) {
        p.smallc = true;
        p.splits = 1;
        return p;
    }
    p.pad = g.pad_small_c();
    p.Cp = p.pad ? g.cpad() : g.C;
    const int M = g.N * g.HO * g.WO, K = g.KH * g.KW * p.Cp;
    p.veck = p.Cp % g.vec() == 0;
    if (p.pad) {
        p.xpad_bytes = align_up((size_t)g.N * g.H * g.W * p.Cp * g.esize());
        p.wpad_bytes = align_up((size_t)g.O * g.KH * g.KW * p.Cp * g.esize());
    }
    if (p.veck) {
        // 8-wave 128 x 256 tiles where there are enough of them to fill the GPU several times
        const bool big = g.O >= 128 && (long long)cdiv(g.O, 128) * cdiv(M, 256) >= 4 * kNumCUs;
        p.cfg = env_override("QLAYER_FWD_CFG", big ? 4 : 3);
        if (p.cfg < 0 || p.cfg >= kFwdCfgs || g.ne != NEURON_QUADRA) p.cfg = 3;  // (the other types: tile 3 only)
        p.BR = kFwdBR[p.cfg];
        p.BCOL = kFwdBCOL[p.cfg];
        p.slots = kFwdSlots[p.cfg];
    } else {
        p.cfg = g.O <= 64 || g.ne != NEURON_QUADRA ? 1 : 0;
        p.BR = p.cfg == 0 ? 128 : 64;
        p.BCOL = 128;
        p.slots = 1;
    }
    p.KE = 64 / (int)g.esize();
    p.row_tiles = cdiv(g.O, p.BR);
    p.col_tiles = cdiv(M, p.BCOL);
    p.stages_total = cdiv(K, p.KE);
    p.ca = p.veck && p.Cp % p.KE == 0 && g.KH * g.KW <= 32 && env_override("QLAYER_FWD_CA", 1) != 0;
    // Position-major order where the maps are small, so that many taps of a
    // position lie in the padding: the splits are planned for the pixel tile
    // with the most in-bounds taps.
    p.pm = p.ca && pm_default(g, env_override("QLAYER_FWD_POSMAJ", -1));
    int kst = p.stages_total;
    if (p.pm) kst = pm_max_taps(g, p.BCOL, M) * (p.Cp / p.KE);
    plan_splits(p.row_tiles * p.col_tiles, kst, 4, (size_t)3 * M * g.O * 4, p.slots, p.splits, p.sps);
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * 3 * M * g.O * sizeof(float)) : 0;
    p.xsq_bytes = g.ne == NEURON_T2 && p.veck ? align_up((size_t)g.N * g.H * g.W * p.Cp * g.esize()) : 0;
    p.ws_bytes = p.xpad_bytes + 3 * p.wpad_bytes + p.part_bytes + p.xsq_bytes;
    return p;
}

// ---------------------------------------------------------------------------
// Input-gradient planning.  Workspace: transposed weights, then split partials.
// ---------------------------------------------------------------------------
// Pipelined input-gradient tile configurations (rows = input channels,
// columns = input pixels):  0: 128 x 128, 1: 64 x 128, 2: 128 x 64, 3: 128 x 128
// with the four waves side by side (each 128 x 32: half the prologue
// products per MFMA of configuration 0), 5: 64 x 128 with the waves side by
// side (each 64 x 32: half the products per MFMA of configuration 1).
constexpr int kBdCfgs = 6;
constexpr int kBdBR[kBdCfgs] = {128, 64, 128, 128, 256, 64};
constexpr int kBdBCOL[kBdCfgs] = {128, 128, 64, 128, 256, 128};  // 4: the wide kernel (8 waves, 16-channel K steps)

struct BwdDataPlan {
    int cfg;  // pipelined: index into kBd*; generic: 0: 128 x 128, 1: 64 x 128
    int BR, BCOL, KE, slots;  // slots: one workgroup per CU (the LDS ring takes 144 KB)
    int row_tiles, col_tiles, splits, sps, stages_total;
    bool veck, s1;
    bool natw;    // weights read untransposed through natural LDS tiles (bf16, C % 8 == 0)
    bool smallc;  // C <= 4: per-pixel partial sums by MFMA, then a gather over the taps
    int fused_rb; // ... stride 1: both steps in one kernel, bands of fused_rb input rows (0: two kernels)
    size_t fused_smem;
    int njb;      // ... 32-column blocks of (r, q, c)
    size_t smem;  // ... LDS of the weight fragments
    size_t wt_bytes, part_bytes, ws_bytes;
};

BwdDataPlan plan_bwd_data(const Geom &g) {
    BwdDataPlan p{};
    {
        const int J = g.KH * g.KW * g.C;  // columns (r, q, c) of the partial sums
        p.njb = cdiv(J, 32);
        p.smem = (size_t)3 * p.njb * (g.O / (2 * g.vec())) * 64 * 16;
        p.smallc = g.C <= 4 && g.O % (2 * g.vec()) == 0 && p.njb <= 2 && p.smem <= 64 * 1024 &&
                   g.ne == NEURON_QUADRA && env_override("QLAYER_BWD_DATA_SMALLC", 1) != 0;
        if (p.smallc) {
            // fused (stride 1): LDS holds the weights and the partial sums of RB + KH - 1
            // output rows; at most 64 KB, so that two workgroups share a CU
            int rb = env_override("QLAYER_BWD_DATA_FUSED_RB", 8);  // (0: the two kernels)
            if (g.SH == 1 && g.SW == 1 && p.njb == 1 && rb > 0) {
                for (; rb >= 1; --rb) {
                    const size_t lds = p.smem + (size_t)(rb + g.KH - 1) * g.WO * kFusedPitch * sizeof(float);
                    if (lds <= 64 * 1024) {
                        p.fused_rb = rb;
                        p.fused_smem = lds;
                        break;
                    }
                }
            }
            p.ws_bytes = p.fused_rb ? 0 : align_up((size_t)g.N * g.HO * g.WO * J * sizeof(float));
            return p;
        }
    }
    const int M = g.N * g.H * g.W, K = g.KH * g.KW * g.O;
    p.veck = g.O % g.vec() == 0;
    p.natw = p.veck && g.dt == QL_BF16 && g.C % 8 == 0;
    p.s1 = g.SH == 1 && g.SW == 1;
    // the wide kernel: bf16, natural weight tiles, stride 1, 16-channel K steps within one tap
    const bool wide_ok = p.natw && p.s1 && g.O % 16 == 0 && g.KH * g.KW <= 32;
    if (p.veck) {
        int dflt = 5;
        if (g.C > 64) dflt = M >= 1024 ? 3 : 2;
        // (measured: faster for 1x1 layers such as the dense layer; for 3x3 layers the
        // 4-wave tiles win, the wide kernel's 8 waves run their product arithmetic in step)
        if (wide_ok && g.KH * g.KW == 1 && g.C >= 256 && M >= 1024) dflt = 4;
        p.cfg = env_override("QLAYER_BWD_DATA_CFG", dflt);
        if (p.cfg < 0 || p.cfg >= kBdCfgs || (p.cfg == 4 && !wide_ok)) p.cfg = 0;
        if (g.ne != NEURON_QUADRA) p.cfg = g.C > 64 ? 3 : 5;  // (the other types: tiles 3 and 5 only)
        p.BR = kBdBR[p.cfg];
        p.BCOL = kBdBCOL[p.cfg];
    } else {
        p.cfg = g.C <= 64 || g.ne != NEURON_QUADRA ? 1 : 0;
        p.BR = p.cfg == 0 ? 128 : 64;
        p.BCOL = 128;
    }
    p.KE = p.cfg == 4 && p.veck ? 16 : 64 / (int)g.esize();
    p.slots = 1;
    p.row_tiles = cdiv(g.C, p.BR);
    p.col_tiles = cdiv(M, p.BCOL);
    p.stages_total = cdiv(K, p.KE);
    plan_splits(p.row_tiles * p.col_tiles, p.stages_total, 4, (size_t)M * g.C * 4, p.slots, p.splits, p.sps);
    p.wt_bytes = p.natw ? 0 : align_up(3 * (size_t)g.O * g.KH * g.KW * g.C * g.esize());
    p.part_bytes = p.splits > 1 ? align_up((size_t)p.splits * M * g.C * sizeof(float)) : 0;
    p.ws_bytes = p.wt_bytes + p.part_bytes;
    return p;
}

// ---------------------------------------------------------------------------
// Weight-gradient planning.  Workspace: dW partials, then db partials.
// ---------------------------------------------------------------------------
// Pipelined (bf16) weight-gradient tile configurations (rows = k', columns =
// output channels per term):  0: 128 x 64, 1: 128 x 128, 2: 64 x 64.
constexpr int kBwCfgs = 3;
constexpr int kBwBKP[kBwCfgs] = {128, 128, 64};
constexpr int kBwBO[kBwCfgs] = {64, 128, 64};
constexpr int kBwSlots[kBwCfgs] = {2, 1, 2};  // workgroups one CU holds at once

struct BwdWeightPlan {
    int cfg;   // pipelined path only
    bool pipe; // bf16 and vectorizable: pipelined kernel; otherwise the generic one
    int BKP, BO, KE, slots;
    int row_tiles, col_tiles, splits, sps, stages_total;
    bool veck;
    bool pad;  // X zero-padded to Cp channels first (pipelined path only)
    int Cp;
    size_t xpad_bytes, dw_bytes, db_bytes, ws_bytes;  // workspace: [X padded][dW partials][db partials]
};

BwdWeightPlan plan_bwd_weight(const Geom &g) {
    BwdWeightPlan p{};
    p.pad = g.dt == QL_BF16 && g.pad_small_c() && g.O % g.vec() == 0;
    p.Cp = p.pad ? g.cpad() : g.C;
    const int M = g.N * g.HO * g.WO, KP = g.KH * g.KW * p.Cp, KPO = g.KH * g.KW * g.C;
    p.veck = p.Cp % g.vec() == 0 && g.O % g.vec() == 0;
    p.pipe = p.veck && g.dt == QL_BF16;
    if (p.pad) p.xpad_bytes = align_up((size_t)g.N * g.H * g.W * p.Cp * g.esize());
    if (p.pipe) {
        p.cfg = env_override("QLAYER_BWD_WEIGHT_CFG", 0);
        if (p.cfg < 0 || p.cfg >= kBwCfgs || g.ne != NEURON_QUADRA) p.cfg = 0;  // (the other types: tile 0)
        p.BKP = kBwBKP[p.cfg];
        p.BO = kBwBO[p.cfg];
        p.slots = kBwSlots[p.cfg];
    } else {
        p.BKP = 128;
        p.BO = 64;
        p.slots = 1;
    }
    p.KE = 64 / (int)g.esize();
    p.row_tiles = cdiv(KP, p.BKP);
    p.col_tiles = cdiv(g.O, p.BO);
    p.stages_total = cdiv(M, p.KE);
    plan_splits(p.row_tiles * p.col_tiles, p.stages_total, env_override("QLAYER_BWD_WEIGHT_MINSTAGES", 16),
                (size_t)3 * g.O * KPO * 4, p.slots, p.splits, p.sps);
    if (p.splits > 1) {
        p.dw_bytes = align_up((size_t)p.splits * 3 * g.O * KPO * sizeof(float));
        p.db_bytes = align_up((size_t)p.splits * 3 * g.O * sizeof(float));
    }
    p.ws_bytes = p.xpad_bytes + p.dw_bytes + p.db_bytes;
    return p;
}

ql_status hip_status() {
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? QL_OK : QL_EHIP;
}

int grid_1d(long long total) {
    long long b = (total + kThreads - 1) / kThreads;
    return (int)std::max(1LL, std::min(b, 8LL * kNumCUs));
}

// ---------------------------------------------------------------------------
// Launch helpers, one per kernel family, dispatching the template instances.
// ---------------------------------------------------------------------------
template <typename T>
ql_status launch_fwd(const Geom &g, const FwdPlan &p, const void *x, const void *wa, const void *wb, const void *wc,
                     const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb, void *ws,
                     const EpiArgs &epi, float *stat_part, hipStream_t st) {
    FwdArgs a{};
    a.epi = epi;
    a.stat_part = stat_part;  // (set by the caller only where the kernel's staged epilogue runs)
    if (p.smallc) {
        a.x = x;
        a.w[0] = wa; a.w[1] = wb; a.w[2] = wc;
        a.bias[0] = ba; a.bias[1] = bb; a.bias[2] = bc;
        a.y = y; a.ta = ta; a.tb = tb;
        a.N = g.N; a.H = g.H; a.W = g.W; a.C = g.C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
        a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
        a.M = g.N * g.HO * g.WO;
        a.K = g.KH * g.KW * g.C;
        a.splits = 1;
        a.fd_howo = make_fastdiv(g.HO * g.WO);
        a.fd_wo = make_fastdiv(g.WO);
        a.fd_c = make_fastdiv(g.C);
        a.fd_kw = make_fastdiv(g.KW);
        a.neuron = g.ne;
        const bool ep = epi.scale || epi.shift || epi.relu;
        // groups of 32 pixels per wave (the next group's loads overlap the current one's stores)
        const long long groups = cdiv(a.M, 32);
        const int gpw = std::max(1, env_override("QLAYER_FWD_SMALLC_GPW", 2));
        const dim3 grid((unsigned)std::max<long long>(
            1, std::min<long long>(cdiv(groups, (long long)(kThreads / 64) * gpw), 4 * kNumCUs)));
#define QL_FWD_SMALLC(OB)                                                                              \
    do {                                                                                               \
        if (ep)                                                                                        \
            hipLaunchKernelGGL((qconv_fwd_smallc_kernel<T, OB, true>), grid, dim3(kThreads), 0, st, a);  \
        else                                                                                           \
            hipLaunchKernelGGL((qconv_fwd_smallc_kernel<T, OB, false>), grid, dim3(kThreads), 0, st, a); \
    } while (0)
        if (g.O == 64) QL_FWD_SMALLC(2);
        else QL_FWD_SMALLC(1);
#undef QL_FWD_SMALLC
        return hip_status();
    }
    a.x = x;
    a.w[0] = wa; a.w[1] = wb; a.w[2] = wc;
    char *wsb = static_cast<char *>(ws);
    if (p.pad) {
        // Zero-pad X and the three weights to Cp channels in the workspace.
        PadSegments sg{};
        const void *srcs[4] = {x, wa, wb, wc};
        const long long wrows = (long long)g.O * g.KH * g.KW;
        const long long rows[4] = {(long long)g.N * g.H * g.W, wrows, g.terms() >= 2 ? wrows : 0,
                                   g.terms() >= 3 ? wrows : 0};  // (terms the type lacks: nothing to pad)
        for (int i = 0; i < 4; ++i) {
            sg.src[i] = srcs[i];
            sg.dst[i] = wsb + (i == 0 ? 0 : p.xpad_bytes + (size_t)(i - 1) * p.wpad_bytes);
            sg.rows[i] = rows[i];
        }
        // (one thread per row when a padded row is one 16-byte vector, else per element)
        const long long pad_items = rows[0] * (p.Cp * (int)sizeof(T) == 16 ? 1 : p.Cp);
        hipLaunchKernelGGL((qconv_pad_channels_kernel<T, 4>), dim3(grid_1d(pad_items), 4), dim3(kThreads), 0, st,
                           sg, g.C, p.Cp);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = sg.dst[0];
        a.w[0] = sg.dst[1]; a.w[1] = sg.dst[2]; a.w[2] = sg.dst[3];
    }
    const int C = p.Cp;  // channels the GEMM sees
    a.bias[0] = ba; a.bias[1] = bb; a.bias[2] = bc;
    a.y = y; a.ta = ta; a.tb = tb;
    a.ws = reinterpret_cast<float *>(wsb + p.xpad_bytes + 3 * p.wpad_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.HO * g.WO;
    a.K = g.KH * g.KW * C;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.fd_howo = make_fastdiv(g.HO * g.WO);
    a.fd_wo = make_fastdiv(g.WO);
    a.fd_c = make_fastdiv(C);
    a.fd_kw = make_fastdiv(g.KW);
    a.pm = p.pm ? 1 : 0;
    a.cps = C / p.KE;
    a.fd_n = make_fastdiv(g.N);
    a.fd_cps = make_fastdiv(std::max(1, a.cps));
    a.neuron = g.ne;
    if (p.xsq_bytes) {
        // T2: X o X once, instead of squaring every fragment in the MFMA loop
        T *xsq = reinterpret_cast<T *>(wsb + p.xpad_bytes + 3 * p.wpad_bytes + p.part_bytes);
        const long long n = (long long)g.N * g.H * g.W * C;
        hipLaunchKernelGGL((qconv_square_kernel<T>), dim3(grid_1d(n / g.vec())), dim3(kThreads), 0, st,
                           static_cast<const T *>(a.x), xsq, n);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = xsq;
        a.xsq = 1;
    }
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    const int om = g.om();
    if (p.veck && om != OM_QUADRA) {
        const bool ca = p.ca;
#define QL_FWD_OM(OM)                                                                                          \
    do {                                                                                                        \
        if (ca)                                                                                                 \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, 64, 128, 2, 2, 4, true, 256, OM>), grid, block, 0, st, a);  \
        else                                                                                                    \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, 64, 128, 2, 2, 4, false, 256, OM>), grid, block, 0, st, a); \
    } while (0)
        if (om == OM_PAIR) QL_FWD_OM(OM_PAIR);
        else if (om == OM_SQUARE) QL_FWD_OM(OM_SQUARE);
        else QL_FWD_OM(OM_SQIN);
#undef QL_FWD_OM
    } else if (!p.veck && om != OM_QUADRA) {
        if (om == OM_PAIR)
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_PAIR>), grid, block, 0, st, a);
        else if (om == OM_SQUARE)
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_SQUARE>), grid, block, 0, st,
                               a);
        else
            hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false, OM_SQIN>), grid, block, 0, st, a);
    } else if (p.veck) {
        // channel-aligned K steps: every step within one tap
        const bool ca = p.ca;
#define QL_FWD(BR, BC, WR, WC, NS, NT)                                                                           \
    do {                                                                                                          \
        if (ca)                                                                                                   \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, BR, BC, WR, WC, NS, true, NT>), grid, dim3(NT), 0, st, a);   \
        else                                                                                                      \
            hipLaunchKernelGGL((qconv_fwd_kernel<T, BR, BC, WR, WC, NS, false, NT>), grid, dim3(NT), 0, st, a);  \
    } while (0)
        switch (p.cfg) {
            case 0: QL_FWD(128, 128, 4, 1, 4, 256); break;
            case 1: QL_FWD(64, 256, 2, 2, 4, 256); break;
            case 2: QL_FWD(128, 128, 2, 2, 4, 256); break;
            case 4: QL_FWD(128, 256, 4, 2, 3, 512); break;
            case 5: QL_FWD(128, 256, 2, 4, 3, 512); break;
            default: QL_FWD(64, 128, 2, 2, 4, 256); break;
        }
#undef QL_FWD
    } else if (p.cfg == 0) {
        hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 128, 128, 2, 2, 64, false>), grid, block, 0, st, a);
    } else {
        hipLaunchKernelGGL((qconv_fwd_generic_kernel<T, 64, 128, 2, 2, 64, false>), grid, block, 0, st, a);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const long long MO = (long long)a.M * g.O;
    if (g.O % 4 == 0)
        hipLaunchKernelGGL((qconv_fwd_combine_kernel<T, true>), dim3(grid_1d(MO / 4)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, MO, g.O, ba, bb, bc, static_cast<T *>(y),
                           static_cast<T *>(ta), static_cast<T *>(tb), g.ne, static_cast<const T *>(x), epi);
    else
        hipLaunchKernelGGL((qconv_fwd_combine_kernel<T, false>), dim3(grid_1d(MO)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, MO, g.O, ba, bb, bc, static_cast<T *>(y),
                           static_cast<T *>(ta), static_cast<T *>(tb), g.ne, static_cast<const T *>(x), epi);
    return hip_status();
}

// Whether launch_fwd's kernel writes Y through its staged epilogue, the path
// that gathers the epilogue statistics itself (qconv_fwd.h).
bool fwd_stats_fused(const Geom &g, const FwdPlan &p) {
    if (p.smallc || !p.veck || p.splits != 1 || g.O % (16 / (int)g.esize()) != 0) return false;
    const int ns = (g.ne == NEURON_QUADRA && (p.cfg == 4 || p.cfg == 5)) ? 3 : 4;
    return fwd_staged_fits(p.BR, p.BCOL, ns, (int)g.esize());
}

template <typename T>
ql_status launch_bwd_data(const Geom &g, const BwdDataPlan &p, const void *gy, const void *ta, const void *tb,
                          const void *wa, const void *wb, const void *wc, void *dx, void *ws, hipStream_t st) {
    if (p.smallc && p.fused_rb) {
        const int bands = cdiv(g.H, p.fused_rb);
#define QL_BD_FUSED(NT)                                                                                            \
    hipLaunchKernelGGL((qconv_bwd_data_cols_fused_kernel<T, NT>), dim3(g.N * bands), dim3(NT), p.fused_smem, st,    \
                       static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),          \
                       static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc),          \
                       static_cast<T *>(dx), g.H, g.W, g.C, g.O, g.KH, g.KW, g.PH, g.PW, g.HO, g.WO, p.fused_rb, \
                       (int)(p.smem / sizeof(v4u)))
        // 8 waves: each takes one or two 32-pixel groups of the band (measured faster than 4)
        if (env_override("QLAYER_BWD_DATA_FUSED_NT", 512) == 256)
            QL_BD_FUSED(256);
        else
            QL_BD_FUSED(512);
#undef QL_BD_FUSED
        return hip_status();
    }
    if (p.smallc) {
        const long long Mo = (long long)g.N * g.HO * g.WO;
        const int J = g.KH * g.KW * g.C;
        float *P = static_cast<float *>(ws);
        const int nblk = cdiv(Mo, 32);
        const dim3 grid(std::max(1, std::min(cdiv(nblk, kThreads / 64), 4 * kNumCUs)));
        if (p.njb == 1)
            hipLaunchKernelGGL((qconv_bwd_data_cols_kernel<T, 1>), grid, dim3(kThreads), p.smem, st,
                               static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),
                               static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc), P,
                               (int)Mo, g.O, g.C, J);
        else
            hipLaunchKernelGGL((qconv_bwd_data_cols_kernel<T, 2>), grid, dim3(kThreads), p.smem, st,
                               static_cast<const T *>(gy), static_cast<const T *>(ta), static_cast<const T *>(tb),
                               static_cast<const T *>(wa), static_cast<const T *>(wb), static_cast<const T *>(wc), P,
                               (int)Mo, g.O, g.C, J);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        const long long M = (long long)g.N * g.H * g.W;
        hipLaunchKernelGGL((qconv_bwd_data_col2im_kernel<T>), dim3(grid_1d(M)), dim3(kThreads), 0, st, P,
                           static_cast<T *>(dx), g.N, g.H, g.W, g.C, g.KH, g.KW, g.SH, g.SW, g.PH, g.PW, g.HO, g.WO);
        return hip_status();
    }
    const int khkw = g.KH * g.KW;
    BwdDataArgs a{};
    ql_status s = QL_OK;
    if (p.natw) {
        a.wt[0] = wa; a.wt[1] = wb; a.wt[2] = wc;
    } else {
        T *wt = static_cast<T *>(ws);
        hipLaunchKernelGGL((qconv_weight_transpose_kernel<T>), dim3(cdiv(g.C, 32), cdiv(g.O, 32), g.terms() * khkw),
                           dim3(kThreads), 0, st, static_cast<const T *>(wa), static_cast<const T *>(wb),
                           static_cast<const T *>(wc), wt, g.O, khkw, g.C);
        s = hip_status();
        if (s != QL_OK) return s;
        const size_t wsz = (size_t)g.O * khkw * g.C;
        a.wt[0] = wt; a.wt[1] = wt + wsz; a.wt[2] = wt + 2 * wsz;
    }
    a.gy = gy; a.ta = ta; a.tb = tb;
    a.dx = dx;
    a.ws = reinterpret_cast<float *>(static_cast<char *>(ws) + p.wt_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = g.C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.H * g.W;
    a.K = khkw * g.O;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.fd_hw = make_fastdiv(g.H * g.W);
    a.fd_w = make_fastdiv(g.W);
    a.fd_o = make_fastdiv(g.O);
    a.fd_kw = make_fastdiv(g.KW);
    a.fd_sh = make_fastdiv(g.SH);
    a.fd_sw = make_fastdiv(g.SW);
    a.neuron = g.ne;
    a.xin = g.ne == NEURON_T2 ? ta : nullptr;  // (T2: the `ta` argument carries X)
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    // channel-aligned K steps (each within one tap): stride 1, natural weight tiles, O a multiple of KE
    const bool bd_ca = p.s1 && p.natw && g.O % p.KE == 0 && g.KH * g.KW <= 32 &&
                       env_override("QLAYER_BWD_DATA_CA", 1) != 0;
    const int om = g.om();
#define QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, NW, OM)                                                                     \
    do {                                                                                                               \
        if (p.s1)                                                                                                      \
            hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, true, NW, false, OM>), grid, block, 0, st, \
                               a);                                                                                     \
        else                                                                                                           \
            hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, false, NW, false, OM>), grid, block, 0,  \
                               st, a);                                                                                 \
    } while (0)
#define QL_BD_PIPE_OM(BR, BCOL, WR, WC, NS, OM)                                                                        \
    do {                                                                                                               \
        if constexpr (sizeof(T) == 2) {                                                                                \
            if (bd_ca) {                                                                                               \
                hipLaunchKernelGGL((qconv_bwd_data_kernel<T, BR, BCOL, WR, WC, NS, true, true, true, OM>), grid, block, \
                                   0, st, a);                                                                          \
                break;                                                                                                 \
            }                                                                                                          \
            if (p.natw) {                                                                                              \
                QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, true, OM);                                                          \
                break;                                                                                                 \
            }                                                                                                          \
        }                                                                                                              \
        QL_BD_PIPE_N(BR, BCOL, WR, WC, NS, false, OM);                                                                 \
    } while (0)
#define QL_BD_PIPE(BR, BCOL, WR, WC, NS) QL_BD_PIPE_OM(BR, BCOL, WR, WC, NS, OM_QUADRA)
#define QL_BD_GEN_OM(BR, BCOL, OM)                                                                                 \
    do {                                                                                                           \
        if (p.s1)                                                                                                  \
            hipLaunchKernelGGL((qconv_bwd_data_generic_kernel<T, BR, BCOL, 2, 2, 64, false, true, OM>), grid, block, \
                               0, st, a);                                                                          \
        else                                                                                                       \
            hipLaunchKernelGGL((qconv_bwd_data_generic_kernel<T, BR, BCOL, 2, 2, 64, false, false, OM>), grid,      \
                               block, 0, st, a);                                                                   \
    } while (0)
#define QL_BD_GEN(BR, BCOL) QL_BD_GEN_OM(BR, BCOL, OM_QUADRA)
#define QL_BD_VARIANT(OM)                                                                                          \
    do {                                                                                                           \
        if (!p.veck)                                                                                               \
            QL_BD_GEN_OM(64, 128, OM);                                                                             \
        else if (p.cfg == 3)                                                                                       \
            QL_BD_PIPE_OM(128, 128, 1, 4, 3, OM);                                                                  \
        else                                                                                                       \
            QL_BD_PIPE_OM(64, 128, 1, 4, 4, OM);                                                                   \
    } while (0)
    if (om == OM_PAIR) {
        QL_BD_VARIANT(OM_PAIR);
    } else if (om == OM_SQUARE) {
        QL_BD_VARIANT(OM_SQUARE);
    } else if (om == OM_SQIN) {
        QL_BD_VARIANT(OM_SQIN);
    } else if (p.veck && p.cfg == 4) {
        if constexpr (sizeof(T) == 2)
            hipLaunchKernelGGL((qconv_bwd_data_wide_kernel<256, 256, 2, 4, 3>), grid, dim3(512), 0, st, a);
    } else if (p.veck) {
        if (p.cfg == 0)
            QL_BD_PIPE(128, 128, 2, 2, 3);
        else if (p.cfg == 1)
            QL_BD_PIPE(64, 128, 2, 2, 4);
        else if (p.cfg == 3)
            QL_BD_PIPE(128, 128, 1, 4, 3);
        else if (p.cfg == 5)
            QL_BD_PIPE(64, 128, 1, 4, 4);
        else
            QL_BD_PIPE(128, 64, 2, 2, 4);
    } else if (p.cfg == 0) {
        QL_BD_GEN(128, 128);
    } else {
        QL_BD_GEN(64, 128);
    }
#undef QL_BD_VARIANT
#undef QL_BD_PIPE
#undef QL_BD_PIPE_OM
#undef QL_BD_PIPE_N
#undef QL_BD_GEN
#undef QL_BD_GEN_OM
    s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const long long total = (long long)a.M * g.C;
    // the neuron type's last step on the summed partials: + G (T4 + identity), x 2 X (T2)
    const int mode = g.ne == NEURON_T4I ? 1 : (g.ne == NEURON_T2 ? 2 : 0);
    const T *src = static_cast<const T *>(mode == 1 ? gy : (mode == 2 ? ta : nullptr));
    if (g.C % 4 == 0)
        hipLaunchKernelGGL((qconv_sum_splits_kernel<T, true>), dim3(grid_1d(total / 4)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, total, static_cast<T *>(dx), mode, src);
    else
        hipLaunchKernelGGL((qconv_sum_splits_kernel<T, false>), dim3(grid_1d(total)), dim3(kThreads), 0, st,
                           static_cast<const float *>(a.ws), p.splits, total, static_cast<T *>(dx), mode, src);
    return hip_status();
}

// The weight-gradient split reduction: dW_t and db_t from the partials
// [split][3][O KH KW C] and [split][3][O], summed in split order.
ql_status reduce_bw_partials(const Geom &g, int splits, const BwdWeightArgs &a, float *dwa, float *dwb, float *dwc,
                             float *dba, float *dbb, float *dbc, hipStream_t st) {
    const long long ndw = (long long)g.O * g.KH * g.KW * g.C;  // dW_t as stored
    if (3 * ndw < (1LL << 20) && splits >= 16 && ndw % 4 == 0)
        hipLaunchKernelGGL(qconv_bwd_weight_reduce2dv_kernel, dim3(grid_1d((3 * ndw / 4 + 3 * g.O) * 16)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else if (3 * ndw < (1LL << 20) && splits >= 16)
        hipLaunchKernelGGL((qconv_bwd_weight_reduce2d_kernel<16>), dim3(grid_1d((3 * ndw + 3 * g.O) * 16)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else if (ndw % 4 == 0)
        hipLaunchKernelGGL((qconv_bwd_weight_reduce_kernel<true>), dim3(grid_1d(3 * ndw / 4 + 3 * g.O)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    else
        hipLaunchKernelGGL((qconv_bwd_weight_reduce_kernel<false>), dim3(grid_1d(3 * ndw + 3 * g.O)),
                           dim3(kThreads), 0, st, static_cast<const float *>(a.ws_dw),
                           static_cast<const float *>(a.ws_db), splits, ndw, g.O, dwa, dwb, dwc, dba, dbb, dbc,
                           a.want_db, g.terms());
    return hip_status();
}

template <typename T>
ql_status launch_bwd_weight(const Geom &g, const BwdWeightPlan &p, const void *x, const void *gy, const void *ta,
                            const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                            void *ws, hipStream_t st) {
    BwdWeightArgs a{};
    a.x = x; a.gy = gy; a.ta = ta; a.tb = tb;
    char *wsb = static_cast<char *>(ws);
    if (p.pad) {
        // Zero-pad X to Cp channels in the workspace; dW_t is stored with the true C.
        PadSegments sg{};
        sg.src[0] = x;
        sg.dst[0] = wsb;
        sg.rows[0] = (long long)g.N * g.H * g.W;
        const long long pad_items = sg.rows[0] * (p.Cp * (int)sizeof(T) == 16 ? 1 : p.Cp);
        hipLaunchKernelGGL((qconv_pad_channels_kernel<T, 1>), dim3(grid_1d(pad_items), 1), dim3(kThreads), 0, st,
                           sg, g.C, p.Cp);
        const ql_status s0 = hip_status();
        if (s0 != QL_OK) return s0;
        a.x = wsb;
    }
    const int C = p.Cp;  // channels the GEMM sees
    a.dw[0] = dwa; a.dw[1] = dwb; a.dw[2] = dwc;
    a.db[0] = dba; a.db[1] = dbb; a.db[2] = dbc;
    a.ws_dw = reinterpret_cast<float *>(wsb + p.xpad_bytes);
    a.ws_db = reinterpret_cast<float *>(wsb + p.xpad_bytes + p.dw_bytes);
    a.zero = zero_page();
    if (!a.zero) return QL_EHIP;
    a.N = g.N; a.H = g.H; a.W = g.W; a.C = C; a.O = g.O; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.M = g.N * g.HO * g.WO;
    a.KP = g.KH * g.KW * C;
    a.C_out = g.C;
    a.row_tiles = p.row_tiles; a.col_tiles = p.col_tiles;
    a.splits = p.splits; a.stages_per_split = p.sps; a.stages_total = p.stages_total;
    a.want_db = dba != nullptr;
    a.fd_howo = make_fastdiv(g.HO * g.WO);
    a.fd_wo = make_fastdiv(g.WO);
    a.fd_c = make_fastdiv(C);
    a.fd_kw = make_fastdiv(g.KW);
    a.lin = g.SH == 1 && g.SW == 1 && g.HO == g.H && g.WO == g.W && env_override("QLAYER_BWD_WEIGHT_LIN", 1) != 0;
    a.lin_dq = (p.KE / g.WO) % g.HO;
    a.lin_dr = p.KE % g.WO;
    a.neuron = g.ne;
    const dim3 grid(p.row_tiles * p.col_tiles * p.splits), block(kThreads);
    const int om = g.om();
    if (om != OM_QUADRA) {
        // the other neuron types: the 128 x 64 pipelined tile (bf16) or the generic 128 x 64 kernel
#define QL_BW_OM(OM)                                                                                               \
    do {                                                                                                           \
        if (p.pipe) {                                                                                              \
            if constexpr (sizeof(T) == 2)                                                                          \
                hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 64, 2, 2, 4, 256, OM>), grid, block, 0, st, a);   \
        } else if (p.veck) {                                                                                       \
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, true, OM>), grid, block, 0, \
                               st, a);                                                                             \
        } else {                                                                                                   \
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, false, OM>), grid, block,   \
                               0, st, a);                                                                          \
        }                                                                                                          \
    } while (0)
        if (om == OM_PAIR) QL_BW_OM(OM_PAIR);
        else if (om == OM_SQUARE) QL_BW_OM(OM_SQUARE);
        else QL_BW_OM(OM_SQIN);
#undef QL_BW_OM
    } else if constexpr (sizeof(T) == 2) {
        if (p.pipe) {
            switch (p.cfg) {
                case 0: hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 64, 2, 2, 4>), grid, block, 0, st, a); break;
                case 1: hipLaunchKernelGGL((qconv_bwd_weight_kernel<128, 128, 2, 2, 4>), grid, block, 0, st, a); break;
                default: hipLaunchKernelGGL((qconv_bwd_weight_kernel<64, 64, 2, 2, 4>), grid, block, 0, st, a); break;
            }
        }
    }
    if (!p.pipe && om == OM_QUADRA) {
        if (p.veck)
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, true>), grid, block, 0, st, a);
        else
            hipLaunchKernelGGL((qconv_bwd_weight_generic_kernel<T, 128, 64, 2, 2, 64, 4, false>), grid, block, 0, st,
                               a);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    return reduce_bw_partials(g, p.splits, a, dwa, dwb, dwc, dba, dbb, dbc, st);
}

// ---------------------------------------------------------------------------
// Depthwise layers (groups == C == O): direct kernels of qconv_depthwise.h.
// 3 x 3 filters at stride 1 or 2 take the column kernels (the input gradient
// at stride 2 the gathering one); other shapes take the generic kernels.
// ---------------------------------------------------------------------------
// Rows per thread of the column kernels and whether they prefetch the next
// column (chosen by measurement on the N=64, C=256, 56x56 layer: the
// configurations that fit the registers without spilling).
constexpr int kDwRowsFwd = 4, kDwRowsBd = 4, kDwRowsBw = 2;

struct DwPlan {
    bool fast;             // 3 x 3 kernels for this pass
    bool col;              // column kernel (else the gathering input-gradient kernel)
    int V;                 // channels per thread (8 or 4)
    bool vec;              // C % V == 0: vector loads
    int lanes, lsh, tiles; // channel lanes per pixel, log2, channel slices
    int R;                 // column kernels: rows per thread
    long long items;       // work items: columns, or input pixels for the gathering kernel
    int ng, iwid;          // column kernels: row groups per image, columns per row
    int ct, tg;            // generic kernels: channel tiles of kDwCB, tap groups of 9
    int splits, pps;       // weight gradient: splits and work items per split
    int grid;              // 3 x 3 forward / input gradient: workgroups (tiles x blocks per slice)
    size_t ws_bytes;
};

int dw_lanes(int C, int V) {
    int l = 1;
    while (l < 8 && l * V < C) l *= 2;
    return l;
}

// pass: 0 forward, 1 input gradient, 2 weight gradient
DwPlan plan_dw(const Geom &g, int pass) {
    DwPlan p{};
    const int taps = g.KH * g.KW;
    // (the 3 x 3 kernels address each tensor with 32-bit buffer offsets)
    const long long xbytes = (long long)g.N * g.H * g.W * g.C * g.esize();
    const long long pbytes = (long long)g.N * g.HO * g.WO * g.C * g.esize();
    p.fast = g.KH == 3 && g.KW == 3 && g.SH == g.SW && g.SH <= 2 && xbytes < (1LL << 31) && pbytes < (1LL << 31);
    p.col = p.fast && (pass != 1 || g.SH == 1);
    // bf16 channel vectors: 16 bytes for the gathering input gradient, else 8
    // (the column kernels' registers; the weight gradient's 27 V accumulators)
    p.V = (g.dt == QL_BF16 && g.C % 8 == 0 && pass == 1 && !p.col) ? 8 : 4;
    p.vec = g.C % p.V == 0;
    p.lanes = dw_lanes(g.C, p.V);
    p.lsh = p.lanes == 1 ? 0 : (p.lanes == 2 ? 1 : (p.lanes == 4 ? 2 : 3));
    p.tiles = cdiv(g.C, p.lanes * p.V);
    p.ct = cdiv(g.C, kDwCB);
    p.tg = cdiv(taps, 9);
    p.R = pass == 0 ? kDwRowsFwd : (pass == 1 ? kDwRowsBd : kDwRowsBw);
    const int rows = pass == 1 ? g.H : g.HO;
    p.iwid = pass == 1 ? g.W : g.WO;
    p.ng = cdiv(rows, p.R);
    p.items = p.col ? (long long)g.N * p.ng * p.iwid : (long long)g.N * (pass == 1 ? g.H * g.W : g.HO * g.WO);
    const int PL = kThreads / p.lanes;
    if (pass != 2) {
        const int chunks = cdiv(p.items, PL);
        const int target = env_override("QLAYER_DW_BLOCKS", 2 * kNumCUs);
        p.grid = p.fast ? std::max(1, std::min(chunks, cdiv(target, p.tiles))) * p.tiles : 0;
        return p;
    }
    // weight gradient: about 2 workgroups per CU, at least 4 items per lane and split
    const long long blocks_per_split = p.fast ? p.tiles : (long long)p.ct * p.tg;
    const int lanes_px = p.fast ? PL : kDwPL;
    p.splits = std::max(1, std::min(cdiv(env_override("QLAYER_DW_BW_BLOCKS", 2 * kNumCUs), blocks_per_split),
                                    cdiv(p.items, (long long)lanes_px * 4)));
    p.pps = cdiv(p.items, p.splits);
    p.splits = cdiv(p.items, p.pps);
    if (p.splits > 1) p.ws_bytes = align_up((size_t)p.splits * 3 * g.C * (taps + 1) * sizeof(float));
    return p;
}

DwArgs dw_args(const Geom &g, const DwPlan &p) {
    DwArgs a{};
    a.N = g.N; a.C = g.C; a.H = g.H; a.W = g.W; a.KH = g.KH; a.KW = g.KW;
    a.SH = g.SH; a.SW = g.SW; a.PH = g.PH; a.PW = g.PW; a.HO = g.HO; a.WO = g.WO;
    a.neuron = g.ne;
    a.J = 3 * g.C * (g.KH * g.KW + 1);
    a.lanes = p.lanes; a.lsh = p.lsh; a.tiles = p.tiles;
    a.ng = p.ng; a.iwid = p.iwid;
    a.fd_howo = make_fastdiv(g.HO * g.WO);
    a.fd_wo = make_fastdiv(g.WO);
    a.fd_hw = make_fastdiv(g.H * g.W);
    a.fd_w = make_fastdiv(g.W);
    a.fd_sh = make_fastdiv(g.SH);
    a.fd_sw = make_fastdiv(g.SW);
    a.fd_item = make_fastdiv(p.ng * p.iwid);
    a.fd_iw = make_fastdiv(p.iwid);
    a.xbytes = (int)std::min<long long>((long long)g.N * g.H * g.W * g.C * g.esize(), INT32_MAX);
    a.pbytes = (int)std::min<long long>((long long)g.N * g.HO * g.WO * g.C * g.esize(), INT32_MAX);
    return a;
}

// 3 x 3 kernels of one operand mode and channel vector.
template <typename T, int OM, int V, bool VEC>
void dw_launch_k(const DwPlan &p, int pass, int S, const DwArgs &a, dim3 grid, size_t smem, hipStream_t st) {
    if (pass == 0) {
        if constexpr (V == 4) {
            if (S == 1) hipLaunchKernelGGL((qconv_dw_fwd_col_kernel<T, OM, V, VEC, 3, 1, kDwRowsFwd, true>), grid, dim3(kThreads), smem, st, a);
            else hipLaunchKernelGGL((qconv_dw_fwd_col_kernel<T, OM, V, VEC, 3, 2, kDwRowsFwd, true>), grid, dim3(kThreads), smem, st, a);
        }
    } else if (pass == 1) {
        // prefetching the next column fits the registers with bf16 only
        constexpr bool PF = sizeof(T) == 2 && V == 4;
        if (!p.col) hipLaunchKernelGGL((qconv_dw_bwd_data_k_kernel<T, OM, V, VEC, 3, 2>), grid, dim3(kThreads), smem, st, a);
        else if constexpr (V == 4) hipLaunchKernelGGL((qconv_dw_bwd_data_col_kernel<T, OM, V, VEC, 3, kDwRowsBd, PF>), grid, dim3(kThreads), smem, st, a);
    } else if constexpr (V == 4) {
        if (S == 1) hipLaunchKernelGGL((qconv_dw_bwd_weight_col_kernel<T, OM, V, VEC, 3, 1, kDwRowsBw>), grid, dim3(kThreads), 0, st, a);
        else hipLaunchKernelGGL((qconv_dw_bwd_weight_col_kernel<T, OM, V, VEC, 3, 2, kDwRowsBw>), grid, dim3(kThreads), 0, st, a);
    }
}
template <typename T, int OM>
void dw_launch_om(const DwPlan &p, int pass, int S, const DwArgs &a, dim3 grid, size_t smem, hipStream_t st) {
    if constexpr (sizeof(T) == 2) {
        if (p.V == 8) return dw_launch_k<T, OM, 8, true>(p, pass, S, a, grid, smem, st);
    }
    if (p.vec) dw_launch_k<T, OM, 4, true>(p, pass, S, a, grid, smem, st);
    else dw_launch_k<T, OM, 4, false>(p, pass, S, a, grid, smem, st);
}
template <typename T>
void dw_launch_fast(const Geom &g, const DwPlan &p, int pass, const DwArgs &a, dim3 grid, size_t smem,
                    hipStream_t st) {
    switch (g.om()) {
        case OM_QUADRA: dw_launch_om<T, OM_QUADRA>(p, pass, g.SH, a, grid, smem, st); break;
        case OM_PAIR: dw_launch_om<T, OM_PAIR>(p, pass, g.SH, a, grid, smem, st); break;
        case OM_SQUARE: dw_launch_om<T, OM_SQUARE>(p, pass, g.SH, a, grid, smem, st); break;
        default: dw_launch_om<T, OM_SQIN>(p, pass, g.SH, a, grid, smem, st); break;
    }
}

// generic kernels: dispatch a template over (T, OM, V4)
#define QL_DW_DISPATCH(KERNEL, EXTRA, GRID, SMEM)                                                              \
    do {                                                                                                       \
        const bool v4 = g.C % 4 == 0;                                                                          \
        const int om = g.om();                                                                                 \
        if (om == OM_QUADRA) {                                                                                 \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_QUADRA, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);    \
            else hipLaunchKernelGGL((KERNEL<T, OM_QUADRA, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
        } else if (om == OM_PAIR) {                                                                            \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_PAIR, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
            else hipLaunchKernelGGL((KERNEL<T, OM_PAIR, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);        \
        } else if (om == OM_SQUARE) {                                                                          \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_SQUARE, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);    \
            else hipLaunchKernelGGL((KERNEL<T, OM_SQUARE, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
        } else {                                                                                               \
            if (v4) hipLaunchKernelGGL((KERNEL<T, OM_SQIN, true EXTRA>), GRID, dim3(kThreads), SMEM, st, a);      \
            else hipLaunchKernelGGL((KERNEL<T, OM_SQIN, false EXTRA>), GRID, dim3(kThreads), SMEM, st, a);        \
        }                                                                                                      \
    } while (0)
#define QL_NOEXTRA
#define QL_TAPS9 , 9

template <typename T>
ql_status launch_dw_fwd(const Geom &g, const void *x, const void *const *w, const float *const *b, void *y,
                        void *ta, void *tb, const EpiArgs &epi, hipStream_t st) {
    const DwPlan p = plan_dw(g, 0);
    DwArgs a = dw_args(g, p);
    a.epi = epi;
    a.x = x;
    for (int t = 0; t < 3; ++t) { a.w[t] = w[t]; a.bias[t] = b[t]; }
    a.y = y; a.yta = ta; a.ytb = tb;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        a.M = (int)p.items;
        const size_t smem = (size_t)g.terms() * (9 + 1) * p.lanes * p.V * sizeof(float);  // filters, biases
        dw_launch_fast<T>(g, p, 0, a, dim3(p.grid), smem, st);
        return hip_status();
    }
    a.M = g.N * g.HO * g.WO;
    const dim3 grid(std::max(1, std::min(cdiv(a.M, kDwPL), cdiv(16 * kNumCUs, p.ct))), p.ct);
    const size_t smem = (size_t)g.terms() * g.KH * g.KW * kDwCB * sizeof(float);
    QL_DW_DISPATCH(qconv_dw_fwd_kernel, QL_NOEXTRA, grid, smem);
    return hip_status();
}

template <typename T>
ql_status launch_dw_bwd_data(const Geom &g, const void *gy, const void *ta, const void *tb, const void *const *w,
                             void *dx, hipStream_t st) {
    const DwPlan p = plan_dw(g, 1);
    DwArgs a = dw_args(g, p);
    a.gy = gy; a.ta = ta; a.tb = tb;
    for (int t = 0; t < 3; ++t) a.w[t] = w[t];
    a.dx = dx;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        a.M = (int)p.items;
        const size_t smem = (size_t)g.terms() * 9 * p.lanes * p.V * sizeof(float);
        dw_launch_fast<T>(g, p, 1, a, dim3(p.grid), smem, st);
        return hip_status();
    }
    a.M = g.N * g.H * g.W;
    const dim3 grid(std::max(1, std::min(cdiv(a.M, kDwPL), cdiv(16 * kNumCUs, p.ct))), p.ct);
    const size_t smem = (size_t)g.terms() * g.KH * g.KW * kDwCB * sizeof(float);
    QL_DW_DISPATCH(qconv_dw_bwd_data_kernel, QL_NOEXTRA, grid, smem);
    return hip_status();
}

template <typename T>
ql_status launch_dw_bwd_weight(const Geom &g, const DwPlan &p, const void *x, const void *gy, const void *ta,
                               const void *tb, float *const *dw, float *const *db, void *ws, hipStream_t st) {
    DwArgs a = dw_args(g, p);
    a.x = x; a.gy = gy; a.ta = ta; a.tb = tb;
    for (int t = 0; t < 3; ++t) { a.dw[t] = dw[t]; a.db[t] = db[t]; }
    a.ws = static_cast<float *>(ws);
    a.splits = p.splits;
    a.px_per_split = p.pps;
    a.M = (int)p.items;
    if (p.fast) {
        a.zero = zero_page();
        if (!a.zero) return QL_EHIP;
        dw_launch_fast<T>(g, p, 2, a, dim3(p.splits, p.tiles), 0, st);
    } else {
        const dim3 grid(p.splits, p.ct, p.tg);
        QL_DW_DISPATCH(qconv_dw_bwd_weight_kernel, QL_TAPS9, grid, 0);
    }
    ql_status s = hip_status();
    if (s != QL_OK || p.splits == 1) return s;
    const int taps = g.KH * g.KW, nt = g.terms();
    const int jn = nt * g.C * taps + (db[0] ? nt * g.C : 0);
    hipLaunchKernelGGL(qconv_dw_reduce_kernel, dim3(cdiv(jn, 16)), dim3(kThreads), 0, st, a.ws, p.splits, a.J, g.C,
                       taps, nt, dw[0], dw[1], dw[2], db[0], db[1], db[2], db[0] != nullptr);
    return hip_status();
}
#undef QL_DW_DISPATCH
#undef QL_NOEXTRA
#undef QL_TAPS9

// The forward epilogue's statistics: partial sums per pixel tile (gathered by
// the staged forward kernel) or per part of rows (a pass over the stored Y'),
// then one reduction in part order.
struct StatPlan {
    bool on, fused;
    int nparts, rpp;  // parts; rows per part of the separate pass
    size_t bytes;
};

StatPlan plan_stats(const Geom &g, const ql_epilogue *e) {
    StatPlan s{};
    s.on = e && e->sum;
    if (!s.on) return s;
    const int M = g.N * g.HO * g.WO;
    FwdPlan p{};
    if (!g.dw) p = plan_fwd(g);
    s.fused = !g.dw && fwd_stats_fused(g, p);
    if (s.fused) {
        s.nparts = p.col_tiles;
    } else {
        s.rpp = std::max(64, cdiv(M, 1024));
        s.nparts = cdiv(M, s.rpp);
    }
    s.bytes = align_up((size_t)s.nparts * 2 * g.O * sizeof(float));
    return s;
}

size_t fwd_ws_bytes(const Geom &g, const ql_epilogue *e) {
    return (g.dw ? 0 : plan_fwd(g).ws_bytes) + plan_stats(g, e).bytes;
}

ql_status fwd_common(const Geom &g, const void *x, const void *wa, const void *wb, const void *wc, const float *ba,
                     const float *bb, const float *bc, void *y, void *ta, void *tb, const ql_epilogue *e, void *ws,
                     size_t ws_bytes, void *stream) {
    const int nt = g.terms();
    // pointers of terms the neuron type lacks are ignored
    if (nt < 3) { wc = nullptr; bc = nullptr; }
    if (nt < 2) { wb = nullptr; bb = nullptr; tb = nullptr; }
    if (g.ne == NEURON_T2) ta = nullptr;  // (nothing is saved: its backward takes X)
    if (!x || !wa || (nt >= 2 && !wb) || (nt >= 3 && !wc)) return QL_EINVAL;
    const bool saved = g.ne == NEURON_T2 ? false : (nt >= 2 ? (ta && tb) : ta != nullptr);
    if (!y && !saved) return QL_EINVAL;
    EpiArgs epi{};
    if (e) {
        // the epilogue transforms Y: it needs Y; the statistics come as a pair
        const bool any = e->scale || e->shift || e->relu || e->sum || e->sumsq;
        if (any && !y) return QL_EINVAL;
        if ((e->sum == nullptr) != (e->sumsq == nullptr)) return QL_EINVAL;
        const void *eps[] = {e->scale, e->shift, e->sum, e->sumsq};
        for (const void *q : eps)
            if (q && !aligned16(q)) return QL_EINVAL;
        epi.scale = e->scale;
        epi.shift = e->shift;
        epi.relu = e->relu != 0;
    }
    const void *ptrs[] = {x, wa, wb, wc, ba, bb, bc, y, ta, tb};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const StatPlan sp = plan_stats(g, e);
    const size_t main_bytes = g.dw ? 0 : plan_fwd(g).ws_bytes;
    if (ws_bytes < main_bytes + sp.bytes || (main_bytes + sp.bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    float *stat_part = sp.on ? reinterpret_cast<float *>(static_cast<char *>(ws) + main_bytes) : nullptr;
    hipStream_t st = static_cast<hipStream_t>(stream);
    ql_status s;
    if (g.dw) {
        const void *w[3] = {wa, wb, wc};
        const float *b[3] = {ba, bb, bc};
        s = g.dt == QL_BF16 ? launch_dw_fwd<uint16_t>(g, x, w, b, y, ta, tb, epi, st)
                            : launch_dw_fwd<float>(g, x, w, b, y, ta, tb, epi, st);
    } else {
        const FwdPlan p = plan_fwd(g);
        float *fused_part = sp.fused ? stat_part : nullptr;
        s = g.dt == QL_BF16
                ? launch_fwd<uint16_t>(g, p, x, wa, wb, wc, ba, bb, bc, y, ta, tb, ws, epi, fused_part, st)
                : launch_fwd<float>(g, p, x, wa, wb, wc, ba, bb, bc, y, ta, tb, ws, epi, fused_part, st);
    }
    if (s != QL_OK || !sp.on) return s;
    const int M = g.N * g.HO * g.WO;
    if (!sp.fused) {
        const dim3 grid(sp.nparts, cdiv(g.O, 64));
        if (g.dt == QL_BF16)
            hipLaunchKernelGGL(qconv_channel_stats_kernel<uint16_t>, grid, dim3(kThreads), 0, st,
                               static_cast<const uint16_t *>(y), M, g.O, sp.rpp, stat_part);
        else
            hipLaunchKernelGGL(qconv_channel_stats_kernel<float>, grid, dim3(kThreads), 0, st,
                               static_cast<const float *>(y), M, g.O, sp.rpp, stat_part);
        s = hip_status();
        if (s != QL_OK) return s;
    }
    hipLaunchKernelGGL(qconv_stats_reduce_kernel, dim3(cdiv(2 * g.O, 4)), dim3(kThreads), 0, st, stat_part,
                       sp.nparts, g.O, e->sum, e->sumsq);
    return hip_status();
}

ql_status bwd_data_common(const Geom &g, const void *gy, const void *ta, const void *tb, const void *wa,
                          const void *wb, const void *wc, void *dx, void *ws, size_t ws_bytes, void *stream) {
    const int nt = g.terms();
    if (nt < 3) wc = nullptr;
    if (nt < 2) wb = nullptr;
    if (g.om() == OM_SQUARE || g.om() == OM_SQIN) tb = nullptr;  // (T2: `ta` is X)
    if (!gy || !ta || !wa || !dx || (nt >= 2 && (!tb || !wb)) || (nt >= 3 && !wc)) return QL_EINVAL;
    const void *ptrs[] = {gy, ta, tb, wa, wb, wc, dx};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    if (g.dw) {
        const void *w[3] = {wa, wb, wc};
        hipStream_t st = static_cast<hipStream_t>(stream);
        return g.dt == QL_BF16 ? launch_dw_bwd_data<uint16_t>(g, gy, ta, tb, w, dx, st)
                               : launch_dw_bwd_data<float>(g, gy, ta, tb, w, dx, st);
    }
    const BwdDataPlan p = plan_bwd_data(g);
    if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return g.dt == QL_BF16 ? launch_bwd_data<uint16_t>(g, p, gy, ta, tb, wa, wb, wc, dx, ws, st)
                           : launch_bwd_data<float>(g, p, gy, ta, tb, wa, wb, wc, dx, ws, st);
}

ql_status bwd_weight_common(const Geom &g, const void *x, const void *gy, const void *ta, const void *tb,
                            float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc, void *ws,
                            size_t ws_bytes, void *stream) {
    const int nt = g.terms(), ngm = om_gmaps(g.om());
    // pointers of terms (and maps) the neuron type lacks are ignored
    if (nt < 3) { dwc = nullptr; dbc = nullptr; }
    if (nt < 2) { dwb = nullptr; dbb = nullptr; }
    if (ngm < 3) tb = nullptr;
    if (ngm < 2) ta = nullptr;
    if (!x || !gy || (ngm >= 2 && !ta) || (ngm >= 3 && !tb) || !dwa || (nt >= 2 && !dwb) || (nt >= 3 && !dwc))
        return QL_EINVAL;
    const int nb = (dba != nullptr) + (dbb != nullptr) + (dbc != nullptr);
    if (nb != 0 && nb != nt) return QL_EINVAL;
    const void *ptrs[] = {x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    if (g.dw) {
        const DwPlan p = plan_dw(g, 2);
        if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
        if (ws && !aligned16(ws)) return QL_EINVAL;
        float *const dw[3] = {dwa, dwb, dwc};
        float *const db[3] = {dba, dbb, dbc};
        hipStream_t st = static_cast<hipStream_t>(stream);
        return g.dt == QL_BF16 ? launch_dw_bwd_weight<uint16_t>(g, p, x, gy, ta, tb, dw, db, ws, st)
                               : launch_dw_bwd_weight<float>(g, p, x, gy, ta, tb, dw, db, ws, st);
    }
    const BwdWeightPlan p = plan_bwd_weight(g);
    if (ws_bytes < p.ws_bytes || (p.ws_bytes && !ws)) return QL_EWORKSPACE;
    if (ws && !aligned16(ws)) return QL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return g.dt == QL_BF16
               ? launch_bwd_weight<uint16_t>(g, p, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, ws, st)
               : launch_bwd_weight<float>(g, p, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, ws, st);
}

}  // namespace

extern "C" {

const char *qlayer_status_string(ql_status s) {
    switch (s) {
        case QL_OK: return "ok";
        case QL_EINVAL: return "invalid argument";
        case QL_EUNSUPPORTED: return "unsupported configuration";
        case QL_EWORKSPACE: return "workspace missing or too small";
        case QL_EHIP: return "HIP runtime error";
    }
    return "unknown status";
}

int qlayer_version(void) { return 100; }

size_t qlayer_conv2d_fwd_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, nullptr);
}

ql_status qlayer_conv2d_fwd(const ql_conv_desc *desc, const void *x, const void *wa, const void *wb, const void *wc,
                            const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb,
                            void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, nullptr, workspace, workspace_bytes, stream);
}

size_t qlayer_conv2d_bwd_data_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    if (g.dw) return 0;
    return plan_bwd_data(g).ws_bytes;
}

ql_status qlayer_conv2d_bwd_data(const ql_conv_desc *desc, const void *gy, const void *ta, const void *tb,
                                 const void *wa, const void *wb, const void *wc, void *dx, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_data_common(g, gy, ta, tb, wa, wb, wc, dx, workspace, workspace_bytes, stream);
}

size_t qlayer_conv2d_bwd_weight_workspace_size(const ql_conv_desc *desc) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    if (g.dw) return plan_dw(g, 2).ws_bytes;
    return plan_bwd_weight(g).ws_bytes;
}

ql_status qlayer_conv2d_bwd_weight(const ql_conv_desc *desc, const void *x, const void *gy, const void *ta,
                                   const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb,
                                   float *dbc, void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return bwd_weight_common(g, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, workspace, workspace_bytes, stream);
}

size_t qlayer_linear_fwd_workspace_size(const ql_linear_desc *desc) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, nullptr);
}

size_t qlayer_conv2d_fwd_ex_workspace_size(const ql_conv_desc *desc, const ql_epilogue *epi) {
    Geom g;
    if (make_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, epi);
}

ql_status qlayer_conv2d_fwd_ex(const ql_conv_desc *desc, const void *x, const void *wa, const void *wb,
                               const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                               void *tb, const ql_epilogue *epi, void *workspace, size_t workspace_bytes,
                               void *stream) {
    Geom g;
    const ql_status s = make_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, epi, workspace, workspace_bytes, stream);
}

size_t qlayer_linear_fwd_ex_workspace_size(const ql_linear_desc *desc, const ql_epilogue *epi) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return fwd_ws_bytes(g, epi);
}

ql_status qlayer_linear_fwd_ex(const ql_linear_desc *desc, const void *x, const void *wa, const void *wb,
                               const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                               void *tb, const ql_epilogue *epi, void *workspace, size_t workspace_bytes,
                               void *stream) {
    Geom g;
    const ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, epi, workspace, workspace_bytes, stream);
}

ql_status qlayer_linear_fwd(const ql_linear_desc *desc, const void *x, const void *wa, const void *wb,
                            const void *wc, const float *ba, const float *bb, const float *bc, void *y, void *ta,
                            void *tb, void *workspace, size_t workspace_bytes, void *stream) {
    Geom g;
    const ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    return fwd_common(g, x, wa, wb, wc, ba, bb, bc, y, ta, tb, nullptr, workspace, workspace_bytes, stream);
}

size_t qlayer_linear_bwd_workspace_size(const ql_linear_desc *desc) {
    Geom g;
    if (linear_geom(desc, g) != QL_OK) return 0;
    return std::max(plan_bwd_data(g).ws_bytes, plan_bwd_weight(g).ws_bytes);
}

ql_status qlayer_linear_bwd(const ql_linear_desc *desc, const void *x, const void *gy, const void *ta,
                            const void *tb, const void *wa, const void *wb, const void *wc, void *dx, float *dwa,
                            float *dwb, float *dwc, float *dba, float *dbb, float *dbc, void *workspace,
                            size_t workspace_bytes, void *stream) {
    Geom g;
    ql_status s = linear_geom(desc, g);
    if (s != QL_OK) return s;
    const int nt = g.terms(), ngm = om_gmaps(g.om());
    // pointers of terms (and maps) the neuron type lacks are ignored
    if (nt < 3) { wc = nullptr; dwc = nullptr; dbc = nullptr; }
    if (nt < 2) { wb = nullptr; dwb = nullptr; dbb = nullptr; }
    if (ngm < 3) tb = nullptr;
    if (ngm < 2) ta = nullptr;
    const int nw = (dwa != nullptr) + (dwb != nullptr) + (dwc != nullptr);
    const int nb = (dba != nullptr) + (dbb != nullptr) + (dbc != nullptr);
    if ((nw != 0 && nw != nt) || (nb != 0 && nb != nt) || (nb != 0 && nw == 0)) return QL_EINVAL;
    if (!dx && nw == 0) return QL_EINVAL;
    if (!x || !gy || (ngm >= 2 && !ta) || (ngm >= 3 && !tb) || !wa || (nt >= 2 && !wb) || (nt >= 3 && !wc))
        return QL_EINVAL;
    // Validate everything before the first launch.
    const void *ptrs[] = {x, gy, ta, tb, wa, wb, wc, dx, dwa, dwb, dwc, dba, dbb, dbc};
    for (const void *q : ptrs)
        if (q && !aligned16(q)) return QL_EINVAL;
    const size_t need = std::max(dx ? plan_bwd_data(g).ws_bytes : 0, nw ? plan_bwd_weight(g).ws_bytes : 0);
    if (workspace_bytes < need || (need && !workspace)) return QL_EWORKSPACE;
    if (dx) {
        // (T2: the input gradient takes X in place of the saved map)
        s = bwd_data_common(g, gy, g.ne == NEURON_T2 ? x : ta, tb, wa, wb, wc, dx, workspace, workspace_bytes, stream);
        if (s != QL_OK) return s;
    }
    if (nw) s = bwd_weight_common(g, x, gy, ta, tb, dwa, dwb, dwc, dba, dbb, dbc, workspace, workspace_bytes, stream);
    return s;
}

}  // extern "C"
