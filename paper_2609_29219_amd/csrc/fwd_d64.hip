// Prefill kernel instantiations, dispatch and resource queries for head
// dimension 64.
#include "common.h"
#include "fwd_kernel.h"

namespace attn {

// Calls F::template run<BN, NW, PIPE, CAUSAL>() for the variant named by the
// runtime values; false if the variant does not exist.
template <typename F>
static bool with_variant(int bn, int waves, int pipe, int causal, F& f) {
#define ATTN_V(BN, NW, PIPE)                                                                   \
    if (bn == BN && waves == NW && pipe == PIPE) {                                             \
        if (causal) f.template run<BN, NW, PIPE, true>();                                      \
        else f.template run<BN, NW, PIPE, false>();                                            \
        return true;                                                                           \
    }
    ATTN_V(32, 4, 0) ATTN_V(32, 4, 1) ATTN_V(32, 8, 0) ATTN_V(32, 8, 1) ATTN_V(32, 8, 2)
    ATTN_V(64, 4, 0) ATTN_V(64, 4, 1) ATTN_V(64, 8, 0) ATTN_V(64, 8, 1) ATTN_V(64, 8, 2)
    ATTN_V(128, 4, 0) ATTN_V(128, 4, 1) ATTN_V(128, 8, 0) ATTN_V(128, 8, 1) ATTN_V(128, 8, 2)
    ATTN_V(32, 4, 3) ATTN_V(32, 8, 3) ATTN_V(64, 4, 3) ATTN_V(64, 8, 3)
#undef ATTN_V
    return false;
}

namespace {
struct Launch {
    const FwdPlan& p;
    const FwdArgs& a;
    hipStream_t st;
    hipError_t err = hipErrorInvalidValue;
    template <int BN, int NW, int PIPE, bool CAUSAL>
    void run() {
        hipLaunchKernelGGL((fwd_kernel<64, BN, NW, PIPE, CAUSAL>), dim3((unsigned)p.grid),
                           dim3(NW * 64), 0, st, a);
        err = hipGetLastError();
    }
};

struct Resources {
    KernelRes* r;
    bool ok = false;
    template <int BN, int NW, int PIPE, bool CAUSAL>
    void run() {
        const void* fn = reinterpret_cast<const void*>(&fwd_kernel<64, BN, NW, PIPE, CAUSAL>);
        hipFuncAttributes a;
        if (hipFuncGetAttributes(&a, fn) != hipSuccess) return;
        int blocks = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, NW * 64, 0) != hipSuccess)
            return;
        r->wg_per_cu = blocks;
        r->scratch_bytes = (int)a.localSizeBytes;
        r->vgprs = a.numRegs;
        ok = true;
    }
};
}  // namespace

hipError_t launch_fwd_d64(const FwdPlan& p, const FwdArgs& a, hipStream_t st) {
    Launch l{p, a, st};
    if (!with_variant(p.block_n, p.waves, p.pipe, p.causal, l)) return hipErrorInvalidValue;
    return l.err;
}

bool fwd_resources_d64(int bn, int waves, int pipe, int causal, KernelRes* r) {
    Resources res{r};
    return with_variant(bn, waves, pipe, causal, res) && res.ok;
}

}  // namespace attn
