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
    int wg_per_cu = 0;
    long long grid = 0;
    double modeled_us = 0.0;
    const char* bound = "";
};

// Candidate domains: every point is an instantiated kernel.
constexpr int kFwdBlockN[] = {32, 64, 128};
constexpr int kFwdWaves[] = {4, 8};
constexpr int kFwdPipe[] = {0, 1, 2, 3};  // 2 only with 8 waves, 3 only with BN <= 64
constexpr int kDecodeThreads = 256;
constexpr int kDecodeUnroll = 8;

// LDS footprint of a prefill workgroup: K tile [BN][D+8] and V tile
// [BN][D+32] in bf16, one slot each (pipe 0) or two (pipe 1, 2, 3).
constexpr int fwd_lds_bytes(int d, int bn, int pipe) {
    return (pipe == 0 ? 1 : 2) * (bn * (d + 8) + bn * (d + 32)) * 2;
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
                    FwdResFn res = nullptr);
// Every feasible candidate (in the planner's search order), up to cap of them
// into out; returns how many there are.
int plan_fwd_all(const attn_device_desc& desc, int B, int H, int Sq, int Skv, int d, int causal,
                 FwdPlan* out, int cap, FwdResFn res = nullptr);
bool fwd_resources(int d, int bn, int waves, int pipe, int causal, KernelRes* out);
bool plan_decode(const attn_device_desc& desc, int B, int Hq, int Hkv, int Skv, int d,
                 int n_splits, DecodePlan* out);
int format_fwd_plan(const FwdPlan& p, char* buf, int buflen);
int format_decode_plan(const DecodePlan& p, char* buf, int buflen);

hipError_t measure_device(attn_device_desc* d);

// Launchers (defined next to the kernels).
hipError_t launch_fwd(const FwdPlan& p, const void* q, const void* k, const void* v, void* o,
                      float* lse, int group, int out_bf16, int Sq, int Skv, float scale,
                      int num_xcds, hipStream_t stream);
hipError_t launch_decode(const DecodePlan& p, const void* q, const void* k, const void* v,
                         float* o, float* lse, float* workspace, int B, int Hq, int Hkv, int Skv,
                         float scale, hipStream_t stream);
// Query heads of one key/value group that a decode workgroup serves together.
int decode_heads_per_wg(int group);

}  // namespace attn
