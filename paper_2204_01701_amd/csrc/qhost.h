// qhost.h -- host-side planning shared by the library's translation units:
// descriptor checks (Geom), tile-configuration and split-K plans, workspace
// sizes, and the launchers each kernel family's translation unit defines.
// Nothing here touches tensor data or allocates device memory.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>

#include "qlayer.h"
#include "qargs.h"
#include "qdevice.h"
#include "qconv_aux.h"
#include "qconv_depthwise.h"
#include "qconv_fwd_smallc.h"
#include "qconv_fwd_narrow.h"

namespace ql {
namespace host {

// Device address of the 16 zero bytes masked-off DMA lanes read (qlayer_api.hip).
const void *zero_page();


constexpr int kNumCUs = 256;         // MI355X compute units
constexpr size_t kAlign = 256;
constexpr long long kMaxElems = (1LL << 31) - 1;  // 32-bit element offsets in the kernels
constexpr size_t kMaxSplitBytes = 128ull << 20;  // cap on split-K partial sums (written + read once)
// Split-K cost model, in units of one K step of one workgroup alone on a CU:
// a CU holding two co-resident workgroups finishes both in kSharedRound steps
// per step each (the second one hides the first one's latency), and one unit
// of time moves about kBytesPerStep bytes of partial sums through HBM.
constexpr double kSharedRound = 1.25;
// ... for the forward kernels, whose second workgroup on a CU adds less (measured on
// the 4 x 4 VGG-16 layers: two splits of 256 workgroups beat four of 512)
constexpr double kSharedRoundFwd = 1.6;
constexpr double kBytesPerStep = 3.2e6;
constexpr double kReduceSteps = 6.0;  // the reduction kernel's launch and ramp
// A workgroup of two pipelines (one per CU) on the two halves of its K range:
// the cost of a K step of each pipeline, in the units above.  The two
// pipelines share the workgroup's barriers, which costs them some of the
// latency hiding of two independent workgroups (measured on the VGG-16
// weight gradients: 1.5 reproduces which of the two kernels is faster on
// every layer).
constexpr double kPipeRound = 1.5;
// A K step of the 8-wave workgroup with the 128-channel tile (one per CU, twice
// the MFMAs of a 64-channel step), in the same units (measured on the same
// layers: 1.2 reproduces where it is the fastest of the three kernels).
constexpr double kFatStep = 1.2;

// Tuning override: QLAYER_<NAME>=<int> replaces a planner choice (for sweeps).
inline int env_override(const char *name, int dflt) {
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    return std::atoi(v);
}

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

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

inline ql_status make_geom(const ql_conv_desc *d, Geom &g) {
    if (!d) return QL_EINVAL;
    if (d->n <= 0 || d->c <= 0 || d->h <= 0 || d->w <= 0 || d->o <= 0 || d->kh <= 0 || d->kw <= 0)
        return QL_EINVAL;
    if (d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0) return QL_EINVAL;
    if (d->dtype != QL_F32 && d->dtype != QL_BF16) return QL_EINVAL;
    if ((int)d->neuron < NEURON_QUADRA || (int)d->neuron > NEURON_T24) return QL_EINVAL;
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
    if (g.dw && g.ne == NEURON_T24) return QL_EUNSUPPORTED;  // (the depthwise kernels cover types 0-4)
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

inline ql_status linear_geom(const ql_linear_desc *d, Geom &g) {
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
inline double plan_splits(int tiles, int stages_total, int min_stages, size_t bytes_per_split, int slots, int &splits,
                          int &sps, size_t max_bytes = kMaxSplitBytes, int pipes = 1,
                          double shared_round = kSharedRound, double step_cost = 1.0) {
    const int cap_bytes = (int)std::max<size_t>(1, max_bytes / std::max<size_t>(bytes_per_split, 1));
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
        double rounds = (double)full * (slots > 1 ? shared_round : 1.0);
        if (rest > 0) rounds += rest > kNumCUs ? shared_round : 1.0;
        double t = per * rounds * step_cost;
        if (pipes > 1) t = (double)cdiv(per, pipes) * (double)(full + (rest > 0)) * kPipeRound;
        if (eff > 1) t += (double)eff * bytes_per_split * 2.0 / kBytesPerStep + kReduceSteps;
        if (s == 1 || t < best) {
            best = t;
            splits = eff;
        }
    }
    sps = cdiv(stages_total, splits);
    splits = cdiv(stages_total, sps);
    return best;
}

// Taps (r, q) in bounds for output position pos = (oh, ow): a bit mask.
inline uint32_t tap_mask(const Geom &g, int pos) {
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
inline int pm_max_taps(const Geom &g, int bcol, long long M) {
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
inline bool pm_default(const Geom &g, int env) {
    if (env >= 0) return env != 0;
    return g.HO * g.WO <= 4 && (g.PH > 0 || g.PW > 0);
}

// Input gradient at stride 1: the taps (r, q) whose output pixel
// (h + PH - r, w + PW - q) lies in the map, for input position pos = h W + w.
inline uint32_t bd_tap_mask(const Geom &g, int pos) {
    const int h = pos / g.W, w = pos % g.W;
    uint32_t u = 0;
    for (int r = 0; r < g.KH; ++r)
        for (int q = 0; q < g.KW; ++q)
            if (h + g.PH - r >= 0 && h + g.PH - r < g.HO && w + g.PW - q >= 0 && w + g.PW - q < g.WO)
                u |= 1u << (r * g.KW + q);
    return u;
}

// The most taps any pixel tile of bcol position-major columns keeps.
inline int bd_pm_max_taps(const Geom &g, int bcol, long long M) {
    int best = 0;
    for (long long m0 = 0; m0 < M; m0 += bcol) {
        const long long m1 = std::min(M, m0 + bcol) - 1;
        uint32_t u = 0;
        for (long long pos = m0 / g.N; pos <= m1 / g.N; ++pos) u |= bd_tap_mask(g, (int)pos);
        best = std::max(best, __builtin_popcount(u));
    }
    return best;
}

// ---------------------------------------------------------------------------
// Forward planning.
// ---------------------------------------------------------------------------
// Pipelined forward tile configurations (rows = output channels per term,
// columns = output pixels; per-wave tile in parentheses; 4 waves unless noted):
//   0: 128 x 128 (32 x 128), 1: 64 x 256 (32 x 128), 2: 128 x 128 (64 x 64), 3: 64 x 128 (32 x 64),
//   4: 128 x 256 (32 x 128, 8 waves), 5: 128 x 256 (64 x 64, 8 waves), 6: as 4 with four LDS stages.
// Larger workgroup tiles move fewer bytes through the vector-memory address
// path per MFMA: 32768 (1/BCOL + 1/(3 BR)) bytes.
constexpr int kFwdCfgs = 7;
constexpr int kFwdBR[kFwdCfgs] = {128, 64, 128, 64, 128, 128, 128};
constexpr int kFwdBCOL[kFwdCfgs] = {128, 256, 128, 128, 256, 256, 256};
// Workgroups one CU holds at once (limited by LDS stages and registers).
constexpr int kFwdSlots[kFwdCfgs] = {1, 1, 1, 2, 1, 1, 1};

// Waves of the narrow kernels (a multiple of the four per workgroup): one per
// 16-pixel block up to three per SIMD, then more blocks per wave.
inline int narrow_waves(long long pixels) {
    const long long waves = std::min<long long>(std::max<long long>(1, cdiv(pixels, 16)), 3LL * 4 * kNumCUs);
    return (int)(cdiv(waves, 4) * 4);
}

struct FwdPlan {
    int cfg;  // pipelined: index into kFwd*; generic: 0: 128 x 128, 1: 64 x 128
    int BR, BCOL, KE, slots;
    int row_tiles, col_tiles, splits, sps, stages_total;
    bool veck;
    bool smallc;  // KH KW C + bias columns <= 32, 32 or 64 output channels: qconv_fwd_smallc_kernel, no workspace
    bool narrow;  // at most 32 output channels, short J: qconv_fwd_narrow_kernel (OB row blocks, NCH chunks)
    int ob, nch;
    bool ksplit;  // small outputs: qconv_fwd_ksplit_kernel (tiles of 3 x 16 krb rows by 16 kcb pixels, K split by waves)
    int krb, kcb;
    int stat_parts;  // partial sums of the epilogue statistics the kernel writes (fused path)
    bool ca;  // channel-aligned K steps (C a multiple of KE, at most 32 taps): every step within one tap
    bool pm;  // position-major pixel order, K steps of padding-only taps skipped (FwdArgs)
    bool pad;                      // X and W_t zero-padded to Cp channels first
    int Cp;
    size_t xpad_bytes, wpad_bytes;  // workspace: [X padded][W_a, W_b, W_c padded][split partials][X o X]
    size_t part_bytes;
    size_t xsq_bytes;               // T2 with 16-byte channel vectors: X o X formed once by a pre-pass
    size_t ws_bytes;
};

inline FwdPlan plan_fwd(const Geom &g) {
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
    // Narrow layers: the weight fragments of all three terms (3 OB NCH runs of
    // 16 bytes per lane) stay in registers for the whole kernel.
    p.ob = cdiv(g.O, 16);
    p.nch = cdiv(K, 4 * g.vec());
    // (one 16-channel row block: two measured slower than the tiled kernel on the
    // 16 -> 32-channel stride-2 layer of a CIFAR ResNet)
    if (p.veck && g.ne == NEURON_QUADRA && g.O % 4 == 0 && p.ob == 1 && p.nch <= 9 &&
        env_override("QLAYER_FWD_NARROW", 1) != 0) {
        p.narrow = true;
        p.splits = 1;
        p.KE = 64 / (int)g.esize();
        p.stat_parts = narrow_waves(M);
        p.ws_bytes = p.xpad_bytes + 3 * p.wpad_bytes;
        return p;
    }
    if (p.veck) {
        // 8-wave 128 x 256 tiles where there are enough of them to fill the GPU several times
        const bool big = g.O >= 128 && (long long)cdiv(g.O, 128) * cdiv(M, 256) >= 4 * kNumCUs;
        // (the 8-wave tile with four stages where the filter has several taps: measured 3 % faster on
        // the N=64, 256-channel 56 x 56 layer, and no faster on the dense layer)
        p.cfg = env_override("QLAYER_FWD_CFG", big ? (g.KH * g.KW > 1 ? 6 : 4) : 3);
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
    p.stat_parts = p.col_tiles;
    p.stages_total = cdiv(K, p.KE);
    // Position-major order where the maps are small, so that many taps of a
    // position lie in the padding: the splits are planned for the pixel tile
    // with the most in-bounds taps.  It needs channel-aligned K steps.  Without
    // it they are on by default in fp32 only: in bf16 they measured slower than
    // the per-lane (r, q, c) addresses (the VGG-16 and CIFAR ResNet layers with
    // 32 to 512 channels and the 256-channel 56 x 56 layer, 2 to 20 %), in fp32
    // 2 to 3 % faster (the ResNet layers with 32 and 64 channels).
    const int ca_env = env_override("QLAYER_FWD_CA", -1);
    const bool pm_want = pm_default(g, env_override("QLAYER_FWD_POSMAJ", -1));
    p.ca = p.veck && p.Cp % p.KE == 0 && g.KH * g.KW <= 32 &&
           (ca_env >= 0 ? ca_env != 0 : (pm_want || g.dt == QL_F32));
    p.pm = p.ca && pm_want;
    int kst = p.stages_total;
    if (p.pm) kst = pm_max_taps(g, p.BCOL, M) * (p.Cp / p.KE);
    plan_splits(p.row_tiles * p.col_tiles, kst, env_override("QLAYER_FWD_MINSTAGES", 4), (size_t)3 * M * g.O * 4,
                p.slots, p.splits, p.sps, kMaxSplitBytes, 1, kSharedRoundFwd);
    // Where these tiles would split K over workgroups (small outputs: the 4 x 4
    // and 2 x 2 maps of a CIFAR VGG-16), the in-workgroup K split of
    // qconv_fwd_ksplit.h instead: tiles small enough to fill the GPU, no
    // partial sums in HBM.  (32-bit byte offsets into X and the weights.)
    // By default only where each wave's K range is at most 768 in bf16 (on
    // longer K the tiled kernel's split-K measured faster: the 512-channel
    // 4 x 4 layers, 1152 per wave, 52 against 47 us per call), 1152 in fp32
    // (the longest measured: the same layers, 215 against 228 us).
    const int ks_env = env_override("QLAYER_FWD_KSPLIT", -1);
    const int ks_k = (pm_want ? pm_max_taps(g, 64, M) : g.KH * g.KW) * p.Cp;
    const int ks_kmax = g.dt == QL_BF16 ? 768 : 1152;
    if (p.veck && g.ne == NEURON_QUADRA && g.O % 4 == 0 && p.Cp % p.KE == 0 && g.KH * g.KW <= 32 &&
        (long long)g.N * g.H * g.W * p.Cp * (long long)g.esize() < (1LL << 31) &&
        (long long)g.O * K * (long long)g.esize() < (1LL << 31) &&
        (ks_env >= 0 ? ks_env != 0 : p.splits > 1 && ks_k <= 4 * ks_kmax)) {
        // the larger tile where its count fills the GPU, else the smaller one (or as forced)
        constexpr int kKsRB[3] = {2, 1, 2}, kKsCB[3] = {4, 4, 2};
        int t = cdiv(g.O, 32) * cdiv(M, 64) >= kNumCUs ? 0 : 1;
        t = env_override("QLAYER_FWD_KSPLIT_TILE", t);
        if (t < 0 || t > 2) t = 1;
        p.ksplit = true;
        p.krb = kKsRB[t];
        p.kcb = kKsCB[t];
        p.pm = pm_want;
        p.row_tiles = cdiv(g.O, 16 * p.krb);
        p.col_tiles = cdiv(M, 16 * p.kcb);
        p.splits = 1;
        p.sps = p.stages_total;
        p.stat_parts = p.col_tiles * p.kcb;
        p.ws_bytes = p.xpad_bytes + 3 * p.wpad_bytes;
        return p;
    }
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
    bool narrow;  // at most 32 input channels, short K: qconv_bwd_data_narrow_kernel (CB row blocks, NCH chunks)
    int cb, nch;
    bool ca, pm;  // channel-aligned K steps; position-major order with taps skipped (BwdDataArgs)
    int order;  // block order of the split-K grid (tile_coord)
    int fused_rb; // ... stride 1: both steps in one kernel, bands of fused_rb input rows (0: two kernels)
    size_t fused_smem;
    int njb;      // ... 32-column blocks of (r, q, c)
    size_t smem;  // ... LDS of the weight fragments
    size_t wt_bytes, part_bytes, ws_bytes;
};

inline BwdDataPlan plan_bwd_data(const Geom &g) {
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
    p.s1 = g.SH == 1 && g.SW == 1;
    // Narrow layers: the transposed weight runs of all three terms stay in registers.
    p.cb = cdiv(g.C, 16);
    p.nch = cdiv(K, 4 * g.vec());
    if (p.veck && g.ne == NEURON_QUADRA && g.C % 4 == 0 && p.cb == 1 && p.nch <= 9 &&
        env_override("QLAYER_BWD_DATA_NARROW", 1) != 0) {
        p.narrow = true;
        p.splits = 1;
        p.wt_bytes = align_up(3 * (size_t)g.O * g.KH * g.KW * g.C * g.esize());
        p.ws_bytes = p.wt_bytes;
        return p;
    }
    p.natw = p.veck && g.dt == QL_BF16 && g.C % 8 == 0;
    // the wide kernel: bf16, natural weight tiles, stride 1, 16-channel K steps within one tap
    const bool wide_ok = p.natw && p.s1 && g.O % 16 == 0 && g.KH * g.KW <= 32;
    if (p.veck) {
        int dflt = 5;
        if (g.C > 64) dflt = M >= 1024 ? 3 : 2;
        // (measured: faster where its 256 x 256 tiles fill the GPU at least twice, as on
        // the dense layer and the N=64, 256-channel 56 x 56 layer; on the small maps of
        // VGG-16 the 4-wave tiles win, the wide kernel's 8 waves run their product
        // arithmetic in step)
        if (wide_ok && g.C >= 256 && (long long)cdiv(g.C, 256) * cdiv(M, 256) >= 2 * kNumCUs) dflt = 4;
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
    // Channel-aligned K steps (each within one tap) in the 4-wave kernels, and
    // with them, on small padded maps, the position-major order that skips
    // the taps whose output pixel lies outside the map for every position of
    // a pixel tile (the proposed neuron: 5 of 9 taps on a 2 x 2 map).
    p.ca = p.s1 && p.natw && p.cfg != 4 && g.O % p.KE == 0 && g.KH * g.KW <= 32 &&
           env_override("QLAYER_BWD_DATA_CA", 1) != 0;
    p.pm = p.ca && g.ne == NEURON_QUADRA && pm_default(g, env_override("QLAYER_BWD_DATA_POSMAJ", -1));
    int kst = p.stages_total;
    if (p.pm) kst = bd_pm_max_taps(g, p.BCOL, M) * (g.O / p.KE);
    plan_splits(p.row_tiles * p.col_tiles, kst, env_override("QLAYER_BWD_DATA_MINSTAGES", 4),
                (size_t)M * g.C * 4, p.slots, p.splits, p.sps);
    // Block order of the split grid: tile-major (each XCD's blocks share pixel
    // tiles: their rows of G, T_a, T_b once, all of the weights) where G, T_a,
    // T_b are at least the weight bytes (M >= C KH KW), split-major otherwise
    // (each XCD reads its K range of the weights and all of G, T_a, T_b).
    // Measured on the VGG-16 layers at batch 128 (bitwise the same results in
    // every order): the 128 -> 256 8 x 8 layer reads 44 instead of 115 MB per
    // call from beyond the L2s and runs 34.0 -> 33.1 us; on the 4 x 4 layers
    // tile-major read twice the bytes (142 against 72 MB per call on 512 ->
    // 512) for at most 1 us, and on the 2 x 2 layers it was 1 us slower.
    {
        const int dflt = (long long)M >= (long long)g.C * g.KH * g.KW ? 1 : 0;
        p.order = p.splits > 1 ? env_override("QLAYER_BWD_DATA_ORDER", dflt) : 0;
        if (p.order < 0 || p.order > 2) p.order = 0;
    }
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
// (3: the 128 x 64 tile of the 16 x 16 x 32 kernel, qconv_bwd_weight16.h;
// 4: the same with two pipelines per 8-wave workgroup; 5: its 128 x 128 tile,
// eight waves side by side in one pipeline)
constexpr int kBwCfgs = 6;
constexpr int kBwBKP[kBwCfgs] = {128, 128, 64, 128, 128, 128};
constexpr int kBwBO[kBwCfgs] = {64, 128, 64, 64, 64, 128};
constexpr int kBwSlots[kBwCfgs] = {2, 1, 2, 2, 1, 1};  // workgroups one CU holds at once
constexpr int kBwThreads[kBwCfgs] = {256, 256, 256, 256, 512, 512};
constexpr int kBwPipes[kBwCfgs] = {1, 1, 1, 1, 2, 1};  // pipelines per workgroup (K halves)

struct BwdWeightPlan {
    bool narrow;  // KH KW C <= 144: qconv_bwd_weight_narrow_kernel (NF fragments, NOB 16-channel slices)
    int nf, nob;
    int cfg;   // pipelined path only
    bool pipe; // bf16 and vectorizable: pipelined kernel; otherwise the generic one
    int BKP, BO, KE, slots;
    int row_tiles, col_tiles, splits, sps, stages_total;
    bool veck;
    bool pad;  // X zero-padded to Cp channels first (pipelined path only)
    int Cp;
    size_t xpad_bytes, dw_bytes, db_bytes, ws_bytes;  // workspace: [X padded][dW partials][db partials]
};

// max_split_bytes: cap on the dW partial sums (the no-allocation entry point
// plans for its fixed scratch array).
inline BwdWeightPlan plan_bwd_weight(const Geom &g, size_t max_split_bytes = kMaxSplitBytes) {
    BwdWeightPlan p{};
    // the narrow kernel: rows k' of at most 144 (after the channel padding)
    const int cp_small = g.pad_small_c() ? g.cpad() : g.C;
    // (wider layers, up to 64 channels, in 16-channel slices, one per workgroup row of the
    // grid: by default in fp32, where the 16 -> 32-channel stride-2 CIFAR ResNet layer
    // measured 37 against 66 us per call; in bf16 it and the VGG-16 stem were no faster)
    const int narrow_max_o = env_override("QLAYER_BWD_WEIGHT_NARROW_MAXO", g.dt == QL_F32 ? 64 : 16);
    const bool narrow_shape = g.ne == NEURON_QUADRA && (g.O <= 16 || (g.O % 16 == 0 && g.O <= narrow_max_o)) &&
                              g.O % g.vec() == 0 && cp_small % g.vec() == 0 &&
                              cdiv(g.KH * g.KW * cp_small, 16) <= 9 &&
                              env_override("QLAYER_BWD_WEIGHT_NARROW", 1) != 0;
    // (fp32 pads only for the narrow kernel)
    p.pad = g.pad_small_c() && g.O % g.vec() == 0 && (g.dt == QL_BF16 || narrow_shape);
    p.Cp = p.pad ? g.cpad() : g.C;
    const int M = g.N * g.HO * g.WO, KP = g.KH * g.KW * p.Cp, KPO = g.KH * g.KW * g.C;
    p.veck = p.Cp % g.vec() == 0 && g.O % g.vec() == 0;
    // pipelined kernels: bf16 every neuron type; fp32 the proposed neuron (the 16 x 16 kernel's fp32 form)
    p.pipe = p.veck && (g.dt == QL_BF16 ||
                        (g.ne == NEURON_QUADRA && env_override("QLAYER_BWD_WEIGHT_F32_PIPE", 1) != 0));
    if (p.pad) p.xpad_bytes = align_up((size_t)g.N * g.H * g.W * p.Cp * g.esize());
    p.KE = 64 / (int)g.esize();
    p.stages_total = cdiv(M, p.KE);
    // (the generic kernel's K steps are latency-bound: splits down to one step
    // each, e.g. the 64 -> 10 head of a CIFAR ResNet at batch 256, 53 -> 17 us)
    const int min_stages = env_override("QLAYER_BWD_WEIGHT_MINSTAGES", p.pipe ? 16 : 1);
    const size_t bytes_per_split = (size_t)3 * g.O * KPO * 4;
    // Narrow layers: the whole gradient of a 16-channel slice is one tile; about
    // two workgroups per CU in all, at least four K steps per wave, the partial
    // sums within max_split_bytes.
    p.nf = cdiv(KP, 16);
    if (narrow_shape && p.Cp == cp_small) {
        p.narrow = true;
        p.nob = cdiv(g.O, 16);
        p.stages_total = cdiv(M, g.dt == QL_BF16 ? 32 : 16);
        int splits = std::min(std::max(1, 2 * kNumCUs / p.nob), std::max(1, cdiv(p.stages_total, 16)));
        splits = env_override("QLAYER_BWD_WEIGHT_NARROW_SPLITS", splits);
        splits = std::max(1, std::min(splits, (int)std::max<size_t>(1, max_split_bytes / bytes_per_split)));
        p.sps = cdiv(p.stages_total, splits);
        p.splits = cdiv(p.stages_total, p.sps);
        if (p.splits > 1) {
            p.dw_bytes = align_up((size_t)p.splits * 3 * g.O * KPO * sizeof(float));
            p.db_bytes = align_up((size_t)p.splits * 3 * g.O * sizeof(float));
        }
        p.ws_bytes = p.xpad_bytes + p.dw_bytes + p.db_bytes;
        return p;
    }
    auto fill = [&](int cfg) {
        p.cfg = cfg;
        p.BKP = p.pipe ? kBwBKP[cfg] : 128;
        p.BO = p.pipe ? kBwBO[cfg] : 64;
        p.slots = p.pipe ? kBwSlots[cfg] : 1;
        p.row_tiles = cdiv(KP, p.BKP);
        p.col_tiles = cdiv(g.O, p.BO);
        return plan_splits(p.row_tiles * p.col_tiles, p.stages_total, min_stages, bytes_per_split, p.slots, p.splits,
                           p.sps, max_split_bytes, kBwPipes[cfg], kSharedRound, cfg == 5 ? kFatStep : 1.0);
    };
    if (p.pipe && g.ne == NEURON_QUADRA) {
        // the 16 x 16 x 32 kernel: four waves on a 64-channel tile, two such pipelines per
        // workgroup, or eight waves on a 128-channel tile, whichever the model finds fastest
        const int forced = env_override("QLAYER_BWD_WEIGHT_CFG", -1);
        if (forced >= (g.dt == QL_BF16 ? 0 : 3) && forced < kBwCfgs) {  // (fp32: configurations 3-5 only)
            fill(forced);
        } else {
            // the 128-channel tile only where it has no empty columns
            const double t3 = fill(3), t4 = fill(4);  // (declarators initialise in order)
            const double t5 = g.O % 128 == 0 ? fill(5) : 1e30;
            const int best = t5 < t3 && t5 < t4 ? 5 : (t4 < t3 ? 4 : 3);
            if (best != 5) fill(best);
        }
    } else {
        fill(0);  // the other neuron types and fp32: the 128 x 64 tile
    }
    if (p.splits > 1) {
        p.dw_bytes = align_up((size_t)p.splits * 3 * g.O * KPO * sizeof(float));
        p.db_bytes = align_up((size_t)p.splits * 3 * g.O * sizeof(float));
    }
    p.ws_bytes = p.xpad_bytes + p.dw_bytes + p.db_bytes;
    return p;
}

inline ql_status hip_status() {
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? QL_OK : QL_EHIP;
}

inline int grid_1d(long long total) {
    long long b = (total + kThreads - 1) / kThreads;
    return (int)std::max(1LL, std::min(b, 8LL * kNumCUs));
}

// ---------------------------------------------------------------------------
// Launch helpers, one per kernel family, dispatching the template instances.
// ---------------------------------------------------------------------------
// Whether launch_fwd's kernel writes Y through its staged epilogue, the path
// that gathers the epilogue statistics itself (qconv_fwd.h).
inline bool fwd_stats_fused(const Geom &g, const FwdPlan &p) {
    if (p.narrow || p.ksplit) return true;
    if (p.smallc || !p.veck || p.splits != 1 || g.O % (16 / (int)g.esize()) != 0) return false;
    const int ns = (g.ne == NEURON_QUADRA && (p.cfg == 4 || p.cfg == 5)) ? 3 : 4;
    return fwd_staged_fits(p.BR, p.BCOL, ns, (int)g.esize());
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

inline int dw_lanes(int C, int V) {
    int l = 1;
    while (l < 8 && l * V < C) l *= 2;
    return l;
}

// pass: 0 forward, 1 input gradient, 2 weight gradient
inline DwPlan plan_dw(const Geom &g, int pass) {
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

inline DwArgs dw_args(const Geom &g, const DwPlan &p) {
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


// ---------------------------------------------------------------------------
// Launchers, one translation unit per kernel family (qlaunch_*.hip): the
// kernels of a call on `st`, dispatched on the dtype.
// ---------------------------------------------------------------------------
ql_status run_fwd(const Geom &g, const FwdPlan &p, const void *x, const void *wa, const void *wb, const void *wc,
                  const float *ba, const float *bb, const float *bc, void *y, void *ta, void *tb, void *ws,
                  const EpiArgs &epi, float *stat_part, hipStream_t st);
// The small-output forward (qlaunch_fwd_ksplit.hip, its own translation unit:
// compiled with the MFMA accumulators in VGPRs) with the arguments run_fwd set up.
template <typename T>
ql_status launch_fwd_ksplit(const FwdPlan &p, const FwdArgs &a, bool ep, hipStream_t st);
ql_status run_bwd_data(const Geom &g, const BwdDataPlan &p, const void *gy, const void *ta, const void *tb,
                       const void *xin, const void *wa, const void *wb, const void *wc, void *dx, void *ws,
                       hipStream_t st);
ql_status run_bwd_weight(const Geom &g, const BwdWeightPlan &p, const void *x, const void *gy, const void *ta,
                         const void *tb, float *dwa, float *dwb, float *dwc, float *dba, float *dbb, float *dbc,
                         void *ws, hipStream_t st);
ql_status run_dw_fwd(const Geom &g, const void *x, const void *const *w, const float *const *b, void *y, void *ta,
                     void *tb, const EpiArgs &epi, hipStream_t st);
ql_status run_dw_bwd_data(const Geom &g, const void *gy, const void *ta, const void *tb, const void *const *w,
                          void *dx, hipStream_t st);
ql_status run_dw_bwd_weight(const Geom &g, const DwPlan &p, const void *x, const void *gy, const void *ta,
                            const void *tb, float *const *dw, float *const *db, void *ws, hipStream_t st);

}  // namespace host
}  // namespace ql

