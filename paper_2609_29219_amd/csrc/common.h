// Internal declarations shared by the translation units of libattn.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn.h"

namespace attn {

// ---------------------------------------------------------------- plans --
// Tile symbols of the prefill kernel, named as the planner reports them.
struct FwdPlan {
    int d = 0;
    int block_m = 0;    // queries per workgroup (32 per wave)
    int block_n = 0;    // keys per K/V tile staged in LDS
    int waves = 0;      // waves per workgroup
    int pipe = 0;       // 0 serial, 1 next tile prefetched, 2 ping-pong wave groups,
                        // 3 software pipeline (softmax between MFMAs)
    int causal = 0;
    int lds_bytes = 0;  // per workgroup
    int vgprs = 0;      // modelled VGPRs per lane
    int wg_per_cu = 0;  // modelled occupancy
    long long grid = 0;
    int n_qtiles = 0;
    int kv_splits = 1;  // key splits per head (non-causal only), with a combine kernel
    int kv_chunk = 0;   // keys per split (a multiple of block_n; Skv when unsplit)
    double modeled_us = 0.0;
    const char* bound = "";  // resource that binds the modelled time
};

// Symbols of the decode pair (partial + combine).
struct DecodePlan {
    int d = 0;
    int n_splits = 0;  // effective split count (every split non-empty)
    int chunk = 0;     // keys per split
    int threads = 0;   // threads per partial workgroup
    int unroll = 0;    // keys per lane group per loop step
    int heads_per_wg = 1;  // query heads of one key/value group served together
    int mfma = 0;          // grouped-query kernel on the matrix cores (16 queries per workgroup)
    int q_blocks = 1;      // query blocks of 16 per key/value head (matrix-core kernel)
    int wg_per_cu = 0;
    long long grid = 0;
    double modeled_us = 0.0;
    const char* bound = "";
};

// Symbols of the GEMM kernel (C = A B, bf16 in, fp32 accumulation).
struct GemmPlan {
    int block_m = 0, block_n = 0, block_k = 0;  // workgroup tile of C and k-step
    int waves_m = 0, waves_n = 0;               // wave grid inside the tile
    int pipe = 0;        // LDS slots - 1: k-tiles in flight while one is multiplied
    int b_nk = 0;        // B stored [N][K] (else [K][N])
    int lds_bytes = 0;
    int vgprs = 0;
    int wg_per_cu = 0;
    int tiles_m = 0, tiles_n = 0;
    // K split (hand-scheduled tiles only): k_splits workgroups per tile each
    // take k_chunk values of k (whole k-tiles; the last split may hold fewer)
    // and write an fp32 partial tile to the workspace; a reduction then sums
    // the partials in split order into C
    int k_splits = 1, k_chunk = 0;
    long long grid = 0;
    double modeled_us = 0.0;
    const char* bound = "";
};

// Workspace bytes of a GEMM plan (the partials of a K split; 0 unsplit).
inline long long gemm_workspace_bytes(const GemmPlan& p, int M, int N) {
    return p.k_splits > 1 ? (long long)p.k_splits * M * N * 4 : 0;
}

// Arguments of one GEMM launch.
struct GemmArgs {
    const uint16_t* a;  // bf16 [M][K]
    const uint16_t* b;  // bf16 [K][N] or [N][K]
    void* c;            // [M][N] fp32 or bf16 (out_bf16)
    int M, N, K;
    int tiles_m, tiles_n;
    int n_wg;
    int num_xcds;
    int out_bf16;
    // K split: workgroup w takes split w / (tiles_m tiles_n) of the grid's
    // split-major order; partial s of C goes to ws + s M N (fp32, [M][N])
    int k_splits;
    int k_chunk;
    float* ws;
};

// Candidate domains: every point is an instantiated kernel.
constexpr int kFwdBlockN[] = {32, 64, 128};
constexpr int kFwdWaves[] = {4, 8};
constexpr int kFwdPipe[] = {0, 1, 2, 3};  // 2 only with 8 waves, 3 only with BN <= 64
constexpr int kDecodeThreads = 256;
constexpr int kDecodeUnroll = 8;
constexpr int kGqaWaves = 4;      // waves of a grouped-query (matrix-core) decode workgroup
constexpr int kGqaMinGroup = 4;   // smallest group served by the matrix-core decode

// Output staging of the prefill epilogue: per wave, 32 rows of one 128-byte
// piece each, padded to 144 bytes (it overlays the K/V slots).
constexpr int kFwdStageRowBytes = 144;
constexpr int kFwdStageWaveBytes = 32 * kFwdStageRowBytes;

// LDS slots of the prefill kernel, in bf16 elements: K tile [BN][D+8] and V
// tile [BN][D+32], each rounded up to whole 1 KiB pieces of the direct
// global-to-LDS tile loads (512 elements).
constexpr int fwd_k_slot_elems(int d, int bn) { return (bn * (d + 8) + 511) / 512 * 512; }
constexpr int fwd_v_slot_elems(int d, int bn) { return (bn * (d + 32) + 511) / 512 * 512; }

// LDS footprint of a prefill workgroup: one K and one V slot (pipe 0) or two
// of each (pipe 1, 2, 3), and at least the waves' output staging.
constexpr int fwd_lds_bytes(int d, int bn, int pipe, int waves) {
    const int slots = (pipe == 0 ? 1 : 2) * (fwd_k_slot_elems(d, bn) + fwd_v_slot_elems(d, bn)) * 2;
    const int stage = waves * kFwdStageWaveBytes;
    return slots > stage ? slots : stage;
}

// Arguments of one prefill launch (every variant takes the same struct).
struct FwdArgs {
    const uint16_t* q;  // bf16 [B][Hq][Sq][D]
    const uint16_t* k;  // bf16 [B][Hkv][Skv][D]
    const uint16_t* v;
    void* o;            // [B][Hq][Sq][D], fp32 or bf16 (out_bf16)
    float* lse;         // [B][Hq][Sq] natural-log log-sum-exp, or null
    int Sq, Skv;
    int n_qtiles;       // q-tiles per head
    int n_wg;           // grid size
    int num_xcds;
    int group;          // query heads per key/value head
    int out_bf16;
    float scale_log2;   // |scale| * log2(e), > 0
    uint32_t q_sign;    // sign bits xor-ed into Q (negative scale)
    // Split key range (non-causal): kv_splits > 1 gives each workgroup the keys
    // [s*kv_chunk, min(Skv, (s+1)*kv_chunk)) of split s, and it writes the
    // unnormalised partials of each row r to index r*kv_splits + s of ws_m
    // (running max, log2 units with the scale), ws_l (sum) and ws_o (d values)
    // instead of o and lse; the split combine then produces o and lse.
    int kv_splits;      // 1: direct output
    int kv_chunk;       // keys per split, a multiple of the tile width (Skv if 1 split)
    float* ws_m;
    float* ws_l;
    float* ws_o;
};

// Resource usage of one compiled prefill variant, as the runtime reports it:
// resident workgroups per CU (registers and LDS together) and private
// (scratch) bytes per lane.  A variant that spills is not a valid primitive.
struct KernelRes {
    int wg_per_cu = 0;
    int scratch_bytes = 0;
    int vgprs = 0;
};
typedef bool (*FwdResFn)(int d, int bn, int waves, int pipe, int causal, KernelRes* out);

// Planner (host only, pure arithmetic on the device description).  With
// res == nullptr (no device) the register footprint is estimated.
void default_desc(attn_device_desc* out);
bool plan_fwd(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d, int causal,
              FwdPlan* out, FwdResFn res = nullptr);
bool plan_fwd_fixed(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d,
                    int causal, int bn, int waves, int pipe, FwdPlan* out,
                    FwdResFn res = nullptr, int kv_splits = 1);
// Key-split counts tried for non-causal prefill (each must leave every split
// non-empty with a chunk that is a multiple of the tile width, and the split
// grid must stay within kFwdSplitRounds rounds of the CUs).
constexpr int kFwdKvSplits[] = {1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 192, 256};
// GEMM K splits (hand-scheduled tiles) and the workspace they may use
constexpr int kGemmKSplits[] = {1, 2, 3, 4, 6, 8};
constexpr long long kGemmMaxWorkspaceBytes = 1LL << 30;
constexpr int kFwdSplitRounds = 4;
// Bytes of the split-KV workspace: rows * splits * (d + 2) floats (the
// partial outputs, then the maxima, then the sums).
inline long long fwd_workspace_bytes(const FwdPlan& p, long long rows) {
    return p.kv_splits > 1 ? rows * p.kv_splits * (p.d + 2) * 4LL : 0;
}
// Every feasible candidate (in the planner's search order), up to cap of them
// into out; returns how many there are.
int plan_fwd_all(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d, int causal,
                 FwdPlan* out, int cap, FwdResFn res = nullptr);
bool fwd_resources(int d, int bn, int waves, int pipe, int causal, KernelRes* out);
// Per-thread switch of the measured per-variant tile costs, prefill and GEMM
// (on by default).
void use_fwd_primitive_costs(bool on);
bool plan_decode(const attn_device_desc& desc, int B, int Hq, int Hkv, int Skv, int d,
                 int n_splits, DecodePlan* out);
// GEMM planner: the same latency model (HEG pipe and for nodes over the
// device description); res, when given, supplies the compiled kernels' real
// footprint.
typedef bool (*GemmResFn)(const GemmPlan& p, KernelRes* out);
bool plan_gemm_fixed(const attn_device_desc& desc, int M, int N, int K, int b_nk, int bm, int bn,
                     int bk, int wm, int wn, int pipe, GemmPlan* out, GemmResFn res = nullptr,
                     int k_splits = 1);
bool plan_gemm(const attn_device_desc& desc, int M, int N, int K, int b_nk, GemmPlan* out,
               GemmResFn res = nullptr);
int plan_gemm_all(const attn_device_desc& desc, int M, int N, int K, int b_nk, GemmPlan* out,
                  int cap, GemmResFn res = nullptr);
bool gemm_resources(const GemmPlan& p, KernelRes* out);
// The 256 x 256 tile on 2 x 2 waves is the hand-scheduled GEMM kernel: it
// runs two to four LDS slots (pipe 1..3) and needs K to be a whole number of
// k-tiles.
inline bool gemm_hand_scheduled(int bm, int bn, int wm, int wn) {
    return bm == 256 && bn == 256 && wm == 2 && wn == 2;
}
int format_gemm_plan(const GemmPlan& p, char* buf, int buflen);
int format_fwd_plan(const FwdPlan& p, char* buf, int buflen);
int format_decode_plan(const DecodePlan& p, char* buf, int buflen);

hipError_t measure_device(attn_device_desc* d);

// Launchers (defined next to the kernels).
// With p.kv_splits > 1, workspace holds fwd_workspace_bytes(p, B*Hq*Sq) bytes
// and a split combine follows the prefill kernel on the same stream.
hipError_t launch_fwd(const FwdPlan& p, const void* q, const void* k, const void* v, void* o,
                      float* lse, int group, int out_bf16, long long rows, int Sq, int Skv,
                      float scale, int num_xcds, float* workspace, hipStream_t stream);
// o[r] = sum_s 2^(m_rs - M) o_rs / sum_s 2^(m_rs - M) l_rs for each of rows rows
// (M = max_s m_rs), fp32 or bf16, and optionally lse[r]; partials at r*n + s.
hipError_t launch_split_combine(int d, const float* ws_m, const float* ws_l, const float* ws_o,
                                void* o, int out_bf16, float* lse, long long rows, int n_splits,
                                hipStream_t stream);
hipError_t launch_decode(const DecodePlan& p, const void* q, const void* k, const void* v,
                         float* o, float* lse, float* workspace, int B, int Hq, int Hkv, int Skv,
                         float scale, int num_xcds, hipStream_t stream);
// With p.k_splits > 1, workspace holds gemm_workspace_bytes(p, M, N) bytes
// and the reduction of the partials follows on the same stream.
hipError_t launch_gemm(const GemmPlan& p, const void* a, const void* b, void* c, int M, int N,
                       int K, int out_bf16, int num_xcds, float* workspace, hipStream_t stream);
// Query heads of one key/value group that a decode workgroup serves together.
int decode_heads_per_wg(int group);

}  // namespace attn
