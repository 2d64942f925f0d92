// Analytic tile/split planner: no autotuning, no measurement in the loop.
//
// The paper keeps block sizes and pipeline knobs symbolic and picks them by
// minimising a latency expression assembled over a Hierarchical Execution
// Graph (HEG) under resource constraints (latency-modelling section:
// sequential composition adds, Eq. heg-seq; a for node multiplies by its
// trip count, Eq. heg-for; a pipe node with load/body/store stages takes a
// sum or a max depending on a two-bit knob, Eq. heg-pipe; the candidate is
// the constrained argmin, Eq. heg-optimization, and the best feasible
// candidate wins, Eq. global-candidate-selection).  The architecture
// description supplies primitive costs and capacities (architecture
// description section).
//
// Here the domain is tiny (3 tile widths x 2 wave counts x 2-3 pipeline
// knob values for prefill; a few dozen split counts for decode), so exhaustive
// enumeration returns the exact argmin a solver would.  The prefill HEG is
//     seq( load Q ; for(n_tiles, pipe(load K/V tile, body, -)) ; store O )
// with body = S = K Q^T, softmax update, O += V^T P^T, and the decode HEG is
//     seq( for(steps, pipe(load K/V keys, local softmax, -)) ; merge ;
//          combine (gather partials, global softmax, final output) ).
// The grid is regular except for causal prefill, whose triangular work is
// regularised by summing per-tile work over the grid plus a tail term (the
// paper's scope paragraph asks for exactly this kind of regularisation).
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>

#include "common.h"
#include "fwd_primitives.inc"
#include "gemm_primitives.inc"

namespace attn {

void default_desc(attn_device_desc* d) {
    memset(d, 0, sizeof *d);
    snprintf(d->arch, sizeof d->arch, "gfx950");
    // structural properties (MI355X specification)
    d->num_cus = 256;
    d->num_xcds = 8;
    d->simds_per_cu = 4;
    d->wave_size = 64;
    d->lds_bytes_per_cu = 160 * 1024;
    d->vgprs_per_simd_lane = 512;
    d->max_waves_per_simd = 8;
    d->clock_ghz = 2.4;
    // performance properties (per-CU primitive rates), as the isolated
    // microbenchmarks of attn_measure_device() measured them on MI355X, in
    // cycles of the nominal clock (the MFMA-bound clock is lower, so the MFMA
    // rate reads below the 4096 flop/clk of the specification)
    d->mfma_bf16_flops_per_clk_cu = 3375.0;
    d->valu_lanes_per_clk_simd = 13.7;
    d->trans_cycles_per_op = 11.9;           // one wave64 v_exp_f32
    d->lds_bytes_per_clk_cu = 135.0;
    d->l2_bytes_per_clk_xcd = 2048.0;
    d->hbm_bytes_per_s = 6.98e12;            // sustained sequential read stream
    d->hbm_latency_us = 2.0;
    d->launch_us = 4.0;
    // prefill resource model, calibrated offline on MI355X (plan_ablation.py
    // --only-calibration --fit: the analytic model alone over every candidate
    // of B2 H16 S4096 d128, non-causal and causal)
    d->issue_cycles_per_score = 66.0;
    d->valu_mfma_overlap = 0.428;
    d->tile_sync_cycles = 220.8;
    d->tile_latency_cycles = 703.8;
}

// HEG composition rules: a pipe node with load, body and store stages and
// the two-bit knob (load/body boundary open, body/store boundary open), and
// a for node repeating its body.
double heg_pipe(double load, double body, double store, int b_lm, int b_ms) {
    if (!b_lm && !b_ms) return load + body + store;
    if (!b_lm && b_ms) return std::max(load + body, store);
    if (b_lm && !b_ms) return std::max(load, body + store);
    return std::max(load, std::max(body, store));
}
double heg_for(double trips, double body) { return trips * body; }

namespace {

int round_up(int x, int a) { return (x + a - 1) / a * a; }

// VGPRs per lane of one prefill wave: Q operand (d/4), score accumulators
// (bn/2; two sets with pipe 3), bf16 probabilities (bn/4), output accumulator
// (d/2), LDS operands in flight (bn/8, plus a deeper ring with pipe 3), one
// source offset per 1 KiB LDS piece the wave loads, staging registers of the
// K and V tiles (pipe 2 only), and scalars/addresses.  Fitted to the compiled
// variants; used only when the compiled kernel cannot be queried.
int fwd_vgprs(int d, int bn, int waves, int pipe) {
    const int nt = waves * 64;
    const int ch = (bn * d / 8 + nt - 1) / nt;
    const int pieces = (bn * ((d + 8) / 8 + (d + 32) / 8) + 63) / 64;
    const int per_wave = (pieces + waves - 1) / waves;
    int v = d / 4 + (pipe == 3 ? 2 : 1) * bn / 2 + bn / 4 + d / 2 + 28 + bn / 8 + per_wave +
            (pipe == 2 ? 2 * ch * 4 : 0) + (pipe == 3 ? 12 : 0);
    return round_up(v, 8);
}

}  // namespace

// Prefill model (cycles of the nominal clock).  Per wave and K/V tile of BN
// keys:
//   M = MFMA cycles: 2*(BN/32)*(D/16) v_mfma_f32_32x32x16_bf16 (S and PV)
//   V = non-MFMA issue cycles: issue_cycles_per_score per score, 32*BN/64
//       scores per lane (softmax VALU, conversions, operand waits)
// With w waves per SIMD (from g resident workgroups of NW waves), a share
// valu_mfma_overlap of V hides behind other waves' MFMAs (none with one wave
// per SIMD), and every workgroup pays tile_sync_cycles per tile:
//   body = g * ((NW/4) * (M + (1 - overlap) * V) + sync)    [ping-pong: 2 syncs]
// LDS bandwidth bounds it from below (K/V operand reads of every wave plus
// the tile writes).  The tile load is a pipe node (load, body, -) whose
// load/body boundary the pipe knob opens (pipe >= 1, Eq. heg-pipe): with pipe
// 0 the load latency is exposed, shared by the g resident workgroups.  A
// q-tile adds one exposed latency (Q and the first tile) to its loop.
//
// Split keys (non-causal, not with the ping-pong schedule; the Flash Decode
// split of the reduction dimension, Evaluation, applied to prefill): with n
// splits every (head, q-tile) becomes n workgroups over chunks of ceil(Skv/n) keys rounded up to whole
// tiles, which fills the CUs when B*H*q-tiles is small; the price is Q read n
// times, the partials (d + 2 floats per row and split) written and read back,
// and a second launch (the split combine, the same global-softmax step as
// decode's).
// Per-variant tile-cost factors (the compiled tile kernels characterised
// once on gfx950, fwd_primitives.inc); a thread may switch them off to see
// the analytic model alone (the calibration script does).
static thread_local bool t_prim_scales = true;
void use_fwd_primitive_costs(bool on) { t_prim_scales = on; }
// GEMM tile kernels: index in kGemmTiles, B layout, pipe, and whether one
// or several workgroups share a CU (a lone workgroup's waves cannot hide
// each other's stalls, so its tiles cost more than the shared-CU model says).
static double gemm_prim_scale(int tile, int b_nk, int pipe, bool shared_cu) {
    constexpr int n_tiles = (int)(sizeof kGemmPrimScale / sizeof kGemmPrimScale[0]);
    constexpr int n_pipes = (int)(sizeof kGemmPrimScale[0][0] / sizeof kGemmPrimScale[0][0][0]);
    if (!t_prim_scales || tile < 0 || tile >= n_tiles || pipe < 0 || pipe >= n_pipes) return 1.0;
    const double f = kGemmPrimScale[tile][b_nk ? 1 : 0][pipe][shared_cu ? 1 : 0];
    return f > 0.0 ? f : 1.0;
}
static double fwd_prim_scale(int d, int bn, int waves, int pipe, int causal) {
    const int di = d == 128 ? 1 : 0;
    const int bi = bn == 32 ? 0 : bn == 64 ? 1 : 2;
    const int wi = waves == 8 ? 1 : 0;
    if (!t_prim_scales || (d != 64 && d != 128) || pipe < 0 || pipe > 3) return 1.0;
    const double f = kFwdPrimScale[di][bi][wi][pipe][causal ? 1 : 0];
    return f > 0.0 ? f : 1.0;
}

bool plan_fwd_fixed(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d,
                    int causal, int bn, int waves, int pipe, FwdPlan* out, FwdResFn res,
                    int kv_splits) {
    FwdPlan p;
    p.d = d;
    p.block_n = bn;
    p.waves = waves;
    p.pipe = pipe;
    p.causal = causal;
    p.block_m = 32 * waves;
    p.lds_bytes = fwd_lds_bytes(d, bn, pipe, waves);
    p.vgprs = fwd_vgprs(d, bn, waves, pipe);
    // legality: capacities and primitive validity
    if (bn % 32 != 0 || d % 32 != 0) return false;
    if (pipe == 2 && waves != 8) return false;
    if (pipe == 3 && bn > 64) return false;
    if (p.lds_bytes > desc.lds_bytes_per_cu) return false;
    if (p.vgprs > desc.vgprs_per_simd_lane) return false;
    const int simds = desc.simds_per_cu;
    const int wpe_regs = desc.vgprs_per_simd_lane / p.vgprs;  // waves per SIMD by registers
    int wg = desc.lds_bytes_per_cu / p.lds_bytes;
    wg = std::min(wg, (wpe_regs * simds) / waves);
    wg = std::min(wg, (desc.max_waves_per_simd * simds) / waves);
    if (res) {  // the compiled kernel's real footprint overrides the estimate
        KernelRes kr;
        if (!res(d, bn, waves, pipe, causal, &kr)) return false;
        if (kr.scratch_bytes > 0) return false;  // spills: not a valid primitive
        wg = kr.wg_per_cu;
        if (kr.vgprs > 0) p.vgprs = kr.vgprs;
    }
    if (wg < 1) return false;
    p.wg_per_cu = wg;
    p.n_qtiles = (Sq + p.block_m - 1) / p.block_m;
    // key splits: every split non-empty, chunks of whole tiles
    if (kv_splits < 1 || (kv_splits > 1 && (causal || pipe == 2))) return false;
    const long long rows = (long long)B * H * Sq;
    p.kv_splits = kv_splits;
    p.kv_chunk = Skv;
    if (kv_splits > 1) {
        const int per = (Skv + kv_splits - 1) / kv_splits;
        p.kv_chunk = (per + bn - 1) / bn * bn;
        if ((Skv + p.kv_chunk - 1) / p.kv_chunk != kv_splits) return false;
        if (rows * d > 0xffffffffLL) return false;  // one combine workgroup per row
    }
    // causal workgroups take q-tile pairs (n-1-u, u)
    p.grid = (long long)B * H * (causal ? (p.n_qtiles + 1) / 2 : (long long)p.n_qtiles * kv_splits);
    if (p.grid > 0x7fffffffLL) return false;
    // splits fill the device; beyond a few rounds of it they only add partials
    if (kv_splits > 1 && p.grid > (long long)kFwdSplitRounds * desc.num_cus) return false;

    const double mfma_cyc = 32768.0 / (desc.mfma_bf16_flops_per_clk_cu / simds);
    const double scores_per_lane = 32.0 * bn / desc.wave_size;
    // ---- primitive costs of one K/V tile -------------------------------
    const double M = 2.0 * (bn / 32) * (d / 16) * mfma_cyc;
    const double V = scores_per_lane * desc.issue_cycles_per_score;
    const double wpw = waves / (double)simds;  // waves of one workgroup per SIMD
    const double syncs = pipe == 2 ? 2.0 : 1.0;
    const double latency = desc.tile_latency_cycles;
    const double prim = fwd_prim_scale(d, bn, waves, pipe, causal);
    // one K/V tile of each of g workgroups resident on a CU: the pipe node
    // (load, body, -), knob b_lm open for pipe >= 1, times the compiled
    // kernel's measured cost relative to this analytic body
    auto tile_cost = [&](int g, double* compute_out, double* lds_out) {
        const double overlap = g * wpw >= 2.0 ? desc.valu_mfma_overlap : 0.0;
        const double compute =
            g * (wpw * (M + (1.0 - overlap) * V) + syncs * desc.tile_sync_cycles);
        const double lds = g * (waves * 4.0 * bn * d + 4.0 * bn * d) / desc.lds_bytes_per_clk_cu;
        if (compute_out) *compute_out = compute;
        if (lds_out) *lds_out = lds;
        return heg_pipe(latency / g, std::max(compute, lds), 0.0, pipe >= 1 ? 1 : 0, 0) * prim;
    };
    double compute = 0.0, lds = 0.0;
    const double tile = tile_cost(wg, &compute, &lds);
    const double load_q = latency;

    // ---- grid: regular (non-causal) or regularised (causal) --------------
    const double slots = (double)desc.num_cus * wg;
    const int chunk_tiles = (p.kv_chunk + bn - 1) / bn;
    double cycles;
    if (!causal) {
        // full rounds of wg workgroups per CU, then a last, partial round in
        // which each CU holds only ceil(tail / CUs) of them (they share the
        // CU with fewer others, so each of its tiles costs less)
        const double full = floor((double)p.grid / slots);
        const double tail = (double)p.grid - full * slots;
        cycles = full * (load_q + heg_for(chunk_tiles, tile));
        if (tail > 0.0) {
            const int r = (int)std::min<double>(wg, ceil(tail / desc.num_cus));
            cycles += load_q + heg_for(chunk_tiles, tile_cost(r, nullptr, nullptr));
        }
    } else {
        // workgroups take q-tile pairs (n-1-u, u), which regularises the
        // triangular work: per workgroup the sum of the pair's tile counts
        auto tiles_of = [&](int qt) {
            const int last_q = std::min(qt * p.block_m + p.block_m - 1, Sq - 1);
            const int kv_end = std::min(Skv, last_q + (Skv - Sq) + 1);
            return (kv_end + bn - 1) / bn;
        };
        // workgroups resident per CU: no more than the grid gives each CU
        // (a grid of one workgroup per CU runs its tiles alone on the CU)
        const int g_eff = (int)std::min<double>(wg, ceil((double)p.grid / desc.num_cus));
        const double tile_c = g_eff == wg ? tile : tile_cost(g_eff, nullptr, nullptr);
        double sum = 0.0, longest = 0.0;
        const int units = (p.n_qtiles + 1) / 2;
        for (int u = 0; u < units; ++u) {
            const int heavy = p.n_qtiles - 1 - u;
            double t = load_q + heg_for(tiles_of(heavy), tile_c);
            if (heavy != u) t += load_q + heg_for(tiles_of(u), tile_c);
            sum += t;
            longest = std::max(longest, t);
        }
        const double rounds = ceil((double)p.grid / ((double)desc.num_cus * g_eff));
        cycles = std::max(rounds * sum / units, longest);
    }
    double us = cycles / (desc.clock_ghz * 1e3);
    // Q read once per split, K/V once, O (or the partials) written once
    const double part_bytes = kv_splits > 1 ? (double)rows * kv_splits * (d + 2) * 4.0 : 0.0;
    const double bytes = (double)B * H * ((double)Sq * d * 2.0 * kv_splits + (double)Skv * d * 4.0) +
                         (kv_splits > 1 ? part_bytes : (double)rows * d * 4.0);
    const double hbm_us = bytes / desc.hbm_bytes_per_s * 1e6;
    // the split combine: a launch, two dependent memory round trips (the
    // maxima, then the sums and outputs), the partials read and O written
    const double combine_us =
        kv_splits > 1 ? desc.launch_us + 2.0 * desc.hbm_latency_us +
                            (part_bytes + (double)rows * d * 4.0) / desc.hbm_bytes_per_s * 1e6 +
                            kv_splits * 0.01
                      : 0.0;
    const char* bound;
    if (hbm_us > us) {
        us = hbm_us;
        bound = "hbm";
    } else if (lds > compute) {
        bound = "lds";
    } else if (pipe == 0 && wg == 1) {
        bound = "latency";
    } else if (M >= (1.0 - (wg * wpw >= 2.0 ? desc.valu_mfma_overlap : 0.0)) * V) {
        bound = "mfma";
    } else {
        bound = "valu";
    }
    p.modeled_us = us + desc.launch_us + combine_us;
    p.bound = bound;
    *out = p;
    return true;
}

bool plan_fwd(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d, int causal,
              FwdPlan* out, FwdResFn res) {
    bool found = false;
    FwdPlan best;
    for (int bn : kFwdBlockN)
        for (int waves : kFwdWaves)
            for (int pipe : kFwdPipe)
                for (int ns : kFwdKvSplits) {
                    FwdPlan p;
                    if (!plan_fwd_fixed(desc, B, H, Sq, Skv, d, causal, bn, waves, pipe, &p, res,
                                        ns))
                        continue;
                    // strict improvement keeps the first (smallest) candidate on ties
                    if (!found || p.modeled_us < best.modeled_us * (1.0 - 1e-9)) {
                        best = p;
                        found = true;
                    }
                }
    if (found) *out = best;
    return found;
}

int plan_fwd_all(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d, int causal,
                 FwdPlan* out, int cap, FwdResFn res) {
    int n = 0;
    for (int bn : kFwdBlockN)
        for (int waves : kFwdWaves)
            for (int pipe : kFwdPipe)
                for (int ns : kFwdKvSplits) {
                    FwdPlan p;
                    if (!plan_fwd_fixed(desc, B, H, Sq, Skv, d, causal, bn, waves, pipe, &p, res,
                                        ns))
                        continue;
                    if (n < cap) out[n] = p;
                    ++n;
                }
    return n;
}

// ------------------------------------------------------------------ GEMM --
// Compiled GEMM tiles (BM, BN, BK, wave grid WM x WN, pipe range); each
// exists for both B layouts and for every pipe setting in its range (pipe + 1
// LDS slots) whose LDS fits.  The 256 x 256 tiles on 2 x 2 waves are the
// hand-scheduled kernel, which needs a second slot.
struct GemmTile {
    int bm, bn, bk, wm, wn, pipe_min, pipe_max;
};
static constexpr int kGemmGroupM = 8;  // tile rows per group of the workgroup order
static constexpr int kGemmPipeMax = 3;
static constexpr GemmTile kGemmTiles[] = {
    {64, 64, 64, 2, 2, 0, 2},    {128, 128, 32, 2, 2, 0, 2}, {128, 128, 64, 2, 2, 0, 2},
    {256, 128, 32, 2, 2, 0, 2},  {256, 128, 64, 2, 2, 0, 2}, {128, 256, 32, 2, 2, 0, 2},
    {128, 256, 64, 2, 2, 0, 2},  {256, 256, 32, 2, 4, 0, 2}, {256, 256, 64, 2, 4, 0, 2},
    {256, 256, 32, 2, 2, 1, 3},  {256, 256, 64, 2, 2, 1, 3},
};
static constexpr int kGemmNumTiles = (int)(sizeof kGemmTiles / sizeof kGemmTiles[0]);

int gemm_lds_bytes(int bm, int bn, int bk, int b_nk, int pipe) {
    const int a = bm * (bk + 8);
    const int b = b_nk ? bn * (bk + 8) : bk * (bn + 32);
    return (pipe + 1) * (a + b) * 2;
}

// The GEMM as an HEG (the paper's GEMM workload with the same latency model
// as the prefill):
//   for(k-tiles, pipe(load, body, -)) per workgroup; workgroups in rounds of
//   (CUs x resident workgroups per CU, g).
// body of one k-tile of one workgroup: the larger of
//   MFMA: 2*BM*BN*BK / mfma_flops_per_clk_cu
//   LDS:  (waves * (MB + NB) * 64 B per k + (BM + BN) * BK * 2) / lds_bytes_per_clk
// g workgroups share the CU: a round (each of them advancing one k-tile)
// takes at least g bodies plus a barrier (tile_sync_cycles).  The load of a
// k-tile takes the latency of where its bytes come from: the tiles resident
// on one XCD share A row panels and B column panels in its L2 (GM tile rows
// per group of the workgroup order), so only the share of the bytes that
// one XCD's resident tiles need once comes from HBM (hbm_latency_us), the
// rest from L2 (tile_latency_cycles).  Pipe knob (Eq. heg-pipe, load/body
// boundary): with pipe 0 the load is exposed, a round takes load + body (or
// g bodies, if longer); with pipe p >= 1, p k-tiles are in flight and a
// round takes the larger of load / p and g bodies.  The HBM bytes of a round
// bound it from below at this CU's share of the HBM bandwidth.  Each
// workgroup adds one exposed load (its first k-tile) and its C store.  This
// is the double-buffering against tile-size trade-off: each extra slot adds
// a tile of LDS, which can cost resident workgroups or rule the largest
// tiles out.  Lower bounds over the whole product: HBM (A, B read once, C
// written once) and L2 (A re-read once per tile column, B once per tile row).
// K split (the same reduction-dimension parallelism as decode's key splits):
// k_splits workgroups per tile each run k_chunk of K (whole k-tiles, no
// split empty) into an fp32 partial, and a reduction sums them: the grid
// grows by k_splits, each workgroup's k-loop shrinks to its chunk, and the
// partials cost their writes and the reduction's launch and traffic.
bool plan_gemm_fixed(const attn_device_desc& desc, int M, int N, int K, int b_nk, int bm, int bn,
                     int bk, int wm, int wn, int pipe, GemmPlan* out, GemmResFn res,
                     int k_splits) {
    int tile_index = -1;
    for (int i = 0; i < kGemmNumTiles; ++i) {
        const GemmTile& t = kGemmTiles[i];
        if (t.bm == bm && t.bn == bn && t.bk == bk && t.wm == wm && t.wn == wn) tile_index = i;
    }
    if (tile_index < 0 || pipe < kGemmTiles[tile_index].pipe_min ||
        pipe > kGemmTiles[tile_index].pipe_max)
        return false;
    if (gemm_hand_scheduled(bm, bn, wm, wn) && K % bk != 0) return false;
    const int n_k_all = (K + bk - 1) / bk;
    if (k_splits < 1 || (k_splits > 1 && !gemm_hand_scheduled(bm, bn, wm, wn))) return false;
    const int chunk_tiles = (n_k_all + k_splits - 1) / k_splits;
    if ((k_splits - 1) * chunk_tiles >= n_k_all) return false;  // a split would be empty
    if (k_splits > 1 && (long long)k_splits * M * N * 4 > kGemmMaxWorkspaceBytes) return false;
    GemmPlan p;
    p.k_splits = k_splits;
    p.k_chunk = k_splits > 1 ? chunk_tiles * bk : K;
    p.block_m = bm;
    p.block_n = bn;
    p.block_k = bk;
    p.waves_m = wm;
    p.waves_n = wn;
    p.pipe = pipe;
    p.b_nk = b_nk ? 1 : 0;
    p.lds_bytes = gemm_lds_bytes(bm, bn, bk, b_nk, pipe);
    const int waves = wm * wn;
    const int mb = bm / (32 * wm), nb = bn / (32 * wn);
    p.vgprs = mb * nb * 16 + 48 + 8 * (mb + nb);  // accumulators, operands, addresses
    if (p.lds_bytes > desc.lds_bytes_per_cu) return false;
    const int simds = desc.simds_per_cu;
    const int wpe_regs = desc.vgprs_per_simd_lane / std::max(p.vgprs, 1);
    int g = desc.lds_bytes_per_cu / p.lds_bytes;
    g = std::min(g, (wpe_regs * simds) / waves);
    g = std::min(g, (desc.max_waves_per_simd * simds) / waves);
    if (res) {
        KernelRes kr;
        if (!res(p, &kr)) return false;
        if (kr.scratch_bytes > 0) return false;  // spills: not a valid primitive
        g = kr.wg_per_cu;
        if (kr.vgprs > 0) p.vgprs = kr.vgprs;
    }
    if (g < 1) return false;
    p.tiles_m = (M + bm - 1) / bm;
    p.tiles_n = (N + bn - 1) / bn;
    p.grid = (long long)p.tiles_m * p.tiles_n * k_splits;
    if (p.grid > 0x7fffffffLL) return false;
    p.wg_per_cu = g;
    // resident workgroups per CU: no more than the grid gives each CU
    const double gr = std::min<double>(g, ceil((double)p.grid / desc.num_cus));

    // ---- one k-tile --------------------------------------------------------
    const double compute = 2.0 * bm * bn * bk / desc.mfma_bf16_flops_per_clk_cu;
    const double lds_bytes = waves * (double)(mb + nb) * 64.0 * bk + (double)(bm + bn) * bk * 2.0;
    const double lds = lds_bytes / desc.lds_bytes_per_clk_cu;
    const double body1 = std::max(compute, lds);
    const double body_g = gr * body1 + desc.tile_sync_cycles;
    // HBM share of a k-tile's bytes: the resident tiles of one XCD need each
    // of their distinct A and B panels once
    const double a_bytes = (double)bm * bk * 2.0, b_bytes = (double)bn * bk * 2.0;
    const double cus_xcd = (double)desc.num_cus / desc.num_xcds;
    const double xcd_tiles = std::max(1.0, std::min((double)p.grid / desc.num_xcds, cus_xcd * gr));
    // the XCD's resident tiles run down groups of kGemmGroupM tile rows: they
    // cover min(tiles_n, resident / GM) columns and the rows that fill them
    const double dn = std::max(1.0, std::min((double)p.tiles_n, ceil(xcd_tiles / kGemmGroupM)));
    const double dm = std::max(1.0, std::min((double)p.tiles_m, ceil(xcd_tiles / dn)));
    const double hbm_per_wg = std::min(a_bytes + b_bytes, (dm * a_bytes + dn * b_bytes) / xcd_tiles);
    const double f_hbm = hbm_per_wg / (a_bytes + b_bytes);
    const double hbm_lat = desc.hbm_latency_us * desc.clock_ghz * 1e3;  // cycles
    const double load = (1.0 - f_hbm) * desc.tile_latency_cycles + f_hbm * hbm_lat;
    const double cu_bw = desc.hbm_bytes_per_s / desc.num_cus / (desc.clock_ghz * 1e9);  // B/clk
    const double t_bw = gr * hbm_per_wg / cu_bw;
    double round = pipe == 0 ? std::max(heg_pipe(load, body1, 0.0, 0, 0), body_g)
                             : heg_pipe(load / pipe, body_g, 0.0, 1, 0);
    round = std::max(round, t_bw);
    const double round_analytic = round;
    // the compiled kernel's measured cost of a k-tile round relative to this
    // analytic one, alone on a CU or sharing it: the factor is measured as a
    // ratio of whole GEMMs of many k-tiles, so it scales the whole round
    // (body, exposed latency and bandwidth alike), not the body alone
    round *= gemm_prim_scale(tile_index, b_nk, pipe, gr >= 2.0);

    const int n_k = chunk_tiles;
    const double store = gr * (double)bm * bn * 4.0 / cu_bw;
    const double rounds = ceil((double)p.grid / (desc.num_cus * gr));
    const double cycles = rounds * (load + heg_for(n_k, round) + store);
    double us = cycles / (desc.clock_ghz * 1e3);
    // C (fp32) once, or each split's partial written and read back plus C
    const double c_bytes = (double)M * N * 4.0 * (k_splits > 1 ? 2.0 * k_splits + 1.0 : 1.0);
    const double hbm_us =
        ((double)M * K * 2.0 + (double)K * N * 2.0 + c_bytes) / desc.hbm_bytes_per_s * 1e6;
    // the reduction: a launch, a dependent memory round trip and its bytes
    const double reduce_us =
        k_splits > 1 ? desc.launch_us + desc.hbm_latency_us +
                           (double)M * N * 4.0 * (k_splits + 1.0) / desc.hbm_bytes_per_s * 1e6
                     : 0.0;
    const double l2_bytes = (double)M * K * 2.0 * p.tiles_n + (double)K * N * 2.0 * p.tiles_m;
    const double l2_us =
        l2_bytes / (desc.l2_bytes_per_clk_xcd * desc.num_xcds * desc.clock_ghz * 1e9) * 1e6;
    const char* bound = lds > compute ? "lds" : "mfma";
    if (round_analytic > body_g) bound = t_bw >= round_analytic ? "hbm" : "latency";
    if (hbm_us > us) {
        us = hbm_us;
        bound = "hbm";
    }
    if (l2_us > us) {
        us = l2_us;
        bound = "l2";
    }
    p.modeled_us = us + desc.launch_us + reduce_us;
    p.bound = bound;
    *out = p;
    return true;
}

int plan_gemm_all(const attn_device_desc& desc, int M, int N, int K, int b_nk, GemmPlan* out,
                  int cap, GemmResFn res) {
    int n = 0;
    for (const GemmTile& t : kGemmTiles)
        for (int pipe = t.pipe_min; pipe <= t.pipe_max; ++pipe)
            for (int splits : kGemmKSplits) {
                GemmPlan p;
                if (!plan_gemm_fixed(desc, M, N, K, b_nk, t.bm, t.bn, t.bk, t.wm, t.wn, pipe, &p,
                                     res, splits))
                    continue;
                if (n < cap) out[n] = p;
                ++n;
            }
    return n;
}

bool plan_gemm(const attn_device_desc& desc, int M, int N, int K, int b_nk, GemmPlan* out,
               GemmResFn res) {
    bool found = false;
    GemmPlan best;
    for (const GemmTile& t : kGemmTiles)
        for (int pipe = t.pipe_min; pipe <= t.pipe_max; ++pipe)
            for (int splits : kGemmKSplits) {
                GemmPlan p;
                if (!plan_gemm_fixed(desc, M, N, K, b_nk, t.bm, t.bn, t.bk, t.wm, t.wn, pipe, &p,
                                     res, splits))
                    continue;
                if (!found || p.modeled_us < best.modeled_us * (1.0 - 1e-9)) {
                    best = p;
                    found = true;
                }
            }
    if (found) *out = best;
    return found;
}

int format_gemm_plan(const GemmPlan& p, char* buf, int buflen) {
    return snprintf(buf, buf ? (size_t)buflen : 0,
                    "kind=gemm BLOCK_M=%d BLOCK_N=%d BLOCK_K=%d WAVES_M=%d WAVES_N=%d PIPE=%d "
                    "K_SPLITS=%d k_chunk=%d b_nk=%d grid=%lld tiles_m=%d tiles_n=%d lds_bytes=%d "
                    "vgprs=%d wg_per_cu=%d modeled_us=%.3f bound=%s",
                    p.block_m, p.block_n, p.block_k, p.waves_m, p.waves_n, p.pipe, p.k_splits,
                    p.k_chunk, p.b_nk, p.grid, p.tiles_m, p.tiles_n, p.lds_bytes, p.vgprs,
                    p.wg_per_cu, p.modeled_us, p.bound);
}

// Query heads per decode workgroup: the largest of 8, 4, 2, 1 dividing the
// number of query heads that share a key/value head.
int decode_heads_per_wg(int group) {
    for (int gq : {8, 4, 2})
        if (group % gq == 0) return gq;
    return 1;
}

bool plan_decode(const attn_device_desc& desc, int B, int Hq, int Hkv, int Skv, int d, int n_req,
                 DecodePlan* out) {
    if (Hkv <= 0 || Hq % Hkv != 0) return false;
    // query heads sharing a key/value head run in one workgroup, which reads
    // each K/V chunk once for all of them.  From kGqaMinGroup heads on, the
    // per-key work is a small dense product and runs on the matrix cores
    // (16 queries per workgroup, 32 keys per wave step, K and V of a step in
    // flight per wave); below, the VALU kernel (GQ heads per workgroup).
    const int group = Hq / Hkv;
    const bool mfma = group >= kGqaMinGroup;
    const int q_blocks = mfma ? (group + 15) / 16 : 1;
    const int gq = mfma ? std::min(group, 16) : decode_heads_per_wg(group);
    const int nt = mfma ? kGqaWaves * 64 : kDecodeThreads;
    const int unroll = mfma ? 1 : (gq >= 4 ? 4 : kDecodeUnroll);
    const int step_keys = mfma ? 32 * kGqaWaves : nt / (d / 8) * unroll;  // keys per loop trip
    // workgroups per split: key/value streams (times query blocks)
    const long long BH = mfma ? (long long)B * Hkv * q_blocks : (long long)B * Hq / gq;
    const long long BHq = (long long)B * Hq;
    const double cu_share = desc.hbm_bytes_per_s / desc.num_cus;  // bytes/s per CU
    int max_wg_cu = std::max(1, desc.max_waves_per_simd * desc.simds_per_cu / (nt / 64));
    if (mfma)  // LDS: one padded 32-key V tile per wave
        max_wg_cu = std::min(max_wg_cu, desc.lds_bytes_per_cu / (kGqaWaves * 32 * (d + 32) * 2 +
                                                                  2 * kGqaWaves * 16 * 4));
    // bytes a workgroup keeps in flight: VALU kernel 2*unroll 16-byte loads
    // per lane; matrix-core kernel one step's K and V per wave
    const double wg_inflight = mfma ? (double)kGqaWaves * 32 * d * 4 : nt * 2.0 * unroll * 16.0;

    auto model = [&](int n, DecodePlan* p) -> bool {
        const int chunk = (Skv + n - 1) / n;
        const int n_eff = (Skv + chunk - 1) / chunk;
        const long long grid = BH * n_eff;
        if (grid > 0x7fffffffLL) return false;
        const double wg_bytes = (double)chunk * d * 4.0;
        const double per_cu = ceil((double)grid / desc.num_cus);  // workgroups per CU
        const double resident = std::min<double>(per_cu, max_wg_cu);
        const double inflight = resident * wg_inflight;  // bytes in flight per CU
        const double cu_bw = std::min(cu_share, inflight / (desc.hbm_latency_us * 1e-6));
        // for(steps, pipe(load, local softmax)): load-bound, loads overlap compute
        const double steps = ceil((double)chunk / step_keys);
        const double stream_us = per_cu * wg_bytes / cu_bw * 1e6;
        const double merge_us = ceil(per_cu / resident) * 1.0;  // LDS merge + write, ~1 us
        // the split combine (a single split writes the output itself)
        const double combine_bytes = (double)BHq * n_eff * (d + 2) * 4.0 + BHq * d * 4.0;
        const double combine_us = n_eff > 1 ? desc.launch_us + 2.0 * desc.hbm_latency_us +
                                                  combine_bytes / desc.hbm_bytes_per_s * 1e6 +
                                                  n_eff * 0.01
                                            : 0.0;
        p->d = d;
        p->n_splits = n_eff;
        p->chunk = chunk;
        p->threads = nt;
        p->unroll = unroll;
        p->heads_per_wg = gq;
        p->mfma = mfma ? 1 : 0;
        p->q_blocks = q_blocks;
        p->wg_per_cu = (int)resident;
        p->grid = grid;
        p->modeled_us = desc.launch_us + stream_us + merge_us + combine_us;
        p->bound = (cu_bw < cu_share) ? "hbm-latency" : "hbm";
        (void)steps;
        return true;
    };

    if (n_req > 0) {
        DecodePlan p;
        if (!model(std::min(n_req, Skv), &p)) return false;
        *out = p;
        return true;
    }
    static const int cand[] = {1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 192, 256, 384, 512};
    bool found = false;
    DecodePlan best;
    for (int n : cand) {
        if (n > 1 && (Skv + n - 1) / n < step_keys) break;  // at least one full step per split
        DecodePlan p;
        if (!model(n, &p)) continue;
        if (!found || p.modeled_us < best.modeled_us * (1.0 - 1e-9)) {
            best = p;
            found = true;
        }
    }
    if (found) *out = best;
    return found;
}

}  // namespace attn

// Internal symbols for unit tests of the composition rules (not part of the
// public header).
extern "C" double attn__heg_pipe(double load, double body, double store, int b_lm, int b_ms) {
    return attn::heg_pipe(load, body, store, b_lm, b_ms);
}
extern "C" double attn__heg_for(double trips, double body) { return attn::heg_for(trips, body); }

namespace attn {

int format_fwd_plan(const FwdPlan& p, char* buf, int buflen) {
    return snprintf(buf, buf ? (size_t)buflen : 0,
                    "kind=fwd d=%d BLOCK_M=%d BLOCK_N=%d WAVES=%d PIPE=%d KV_SPLITS=%d "
                    "KV_CHUNK=%d causal=%d grid=%lld n_qtiles=%d lds_bytes=%d vgprs=%d "
                    "wg_per_cu=%d modeled_us=%.3f bound=%s",
                    p.d, p.block_m, p.block_n, p.waves, p.pipe, p.kv_splits, p.kv_chunk,
                    p.causal, p.grid, p.n_qtiles, p.lds_bytes, p.vgprs, p.wg_per_cu,
                    p.modeled_us, p.bound);
}

int format_decode_plan(const DecodePlan& p, char* buf, int buflen) {
    return snprintf(buf, buf ? (size_t)buflen : 0,
                    "kind=decode d=%d N_SPLITS=%d CHUNK=%d THREADS=%d UNROLL=%d HEADS_PER_WG=%d "
                    "MFMA=%d Q_BLOCKS=%d grid=%lld wg_per_cu=%d modeled_us=%.3f bound=%s",
                    p.d, p.n_splits, p.chunk, p.threads, p.unroll, p.heads_per_wg, p.mfma,
                    p.q_blocks, p.grid, p.wg_per_cu, p.modeled_us, p.bound);
}

}  // namespace attn
