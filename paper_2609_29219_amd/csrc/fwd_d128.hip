// Prefill kernel instantiations and dispatch for head dimension 128.
#include "common.h"
#include "fwd_kernel.h"

namespace attn {

template <int BN, int NW, bool DBUF, bool CAUSAL>
static hipError_t launch_one(const FwdPlan& p, const void* q, const void* k, const void* v,
                             float* o, int Sq, int Skv, float scale_log2, uint32_t q_sign,
                             int num_xcds, hipStream_t stream) {
    hipLaunchKernelGGL((fwd_kernel<128, BN, NW, DBUF, CAUSAL>), dim3((unsigned)p.grid),
                       dim3(NW * 64), 0, stream, static_cast<const uint16_t*>(q),
                       static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), o, Sq,
                       Skv, p.n_qtiles, (int)p.grid, num_xcds, scale_log2, q_sign);
    return hipGetLastError();
}

template <int BN, int NW>
static hipError_t launch_bn_nw(const FwdPlan& p, const void* q, const void* k, const void* v,
                               float* o, int Sq, int Skv, float sl, uint32_t qs, int nx,
                               hipStream_t st) {
    if (p.dbuf) {
        return p.causal ? launch_one<BN, NW, true, true>(p, q, k, v, o, Sq, Skv, sl, qs, nx, st)
                        : launch_one<BN, NW, true, false>(p, q, k, v, o, Sq, Skv, sl, qs, nx, st);
    }
    return p.causal ? launch_one<BN, NW, false, true>(p, q, k, v, o, Sq, Skv, sl, qs, nx, st)
                    : launch_one<BN, NW, false, false>(p, q, k, v, o, Sq, Skv, sl, qs, nx, st);
}

hipError_t launch_fwd_d128(const FwdPlan& p, const void* q, const void* k, const void* v,
                            float* o, int Sq, int Skv, float scale_log2, uint32_t q_sign,
                            int num_xcds, hipStream_t st) {
#define ATTN_CASE(BN, NW)                                                                   \
    if (p.block_n == BN && p.waves == NW)                                                   \
        return launch_bn_nw<BN, NW>(p, q, k, v, o, Sq, Skv, scale_log2, q_sign, num_xcds, st);
    ATTN_CASE(32, 4)
    ATTN_CASE(32, 8)
    ATTN_CASE(64, 4)
    ATTN_CASE(64, 8)
    ATTN_CASE(128, 4)
    ATTN_CASE(128, 8)
#undef ATTN_CASE
    return hipErrorInvalidValue;
}

template <int BN, int NW, bool DBUF, bool CAUSAL>
static bool resources_one(KernelRes* r) {
    const void* fn = reinterpret_cast<const void*>(&fwd_kernel<128, BN, NW, DBUF, CAUSAL>);
    hipFuncAttributes a;
    if (hipFuncGetAttributes(&a, fn) != hipSuccess) return false;
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, NW * 64, 0) != hipSuccess)
        return false;
    r->wg_per_cu = blocks;
    r->scratch_bytes = (int)a.localSizeBytes;
    r->vgprs = a.numRegs;
    return true;
}

bool fwd_resources_d128(int bn, int waves, int dbuf, int causal, KernelRes* r) {
#define ATTN_RES(BN, NW)                                                                     \
    if (bn == BN && waves == NW) {                                                           \
        if (dbuf) return causal ? resources_one<BN, NW, true, true>(r)                      \
                                : resources_one<BN, NW, true, false>(r);                    \
        return causal ? resources_one<BN, NW, false, true>(r)                               \
                      : resources_one<BN, NW, false, false>(r);                             \
    }
    ATTN_RES(32, 4)
    ATTN_RES(32, 8)
    ATTN_RES(64, 4)
    ATTN_RES(64, 8)
    ATTN_RES(128, 4)
    ATTN_RES(128, 8)
#undef ATTN_RES
    return false;
}

}  // namespace attn
