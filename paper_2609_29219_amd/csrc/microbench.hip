// Microbenchmarks that measure the performance properties of the device
// description (the paper's architecture-description section: structural
// properties come from the specification, performance properties from
// isolated microbenchmarks, measured a single time per architecture and used for
// every shape).  Each kernel saturates one primitive on every CU:
//   mfma  -- independent v_mfma_f32_32x32x16_bf16 chains, 4 waves per CU
//   valu  -- independent fp32 FMA chains
//   trans -- independent v_exp_f32 chains
//   lds   -- conflict-free ds_read_b128 streams
//   hbm   -- a grid-stride 16-byte read stream over a large buffer
// Rates are converted to per-clock figures with the engine clock the
// runtime reports.
#include <math.h>
#include <string.h>

#include "common.h"

namespace attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void mb_mfma(float* out, int iters) {
    const int l = threadIdx.x;
    bf16x8 a, b;
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(float)((l + e) & 7);
        b[e] = (__bf16)(float)((l * 3 + e) & 7);
    }
    f32x16 acc[kChains];
    for (int c = 0; c < kChains; ++c)
        for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
    for (int i = 0; i < iters; ++i)
#pragma unroll
        for (int c = 0; c < kChains; ++c)
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    float s = 0.f;
    for (int c = 0; c < kChains; ++c)
        for (int r = 0; r < 16; ++r) s += acc[c][r];
    out[blockIdx.x * blockDim.x + l] = s;
}

__global__ __launch_bounds__(256) void mb_valu(float* out, int iters, float a, float b) {
    float x[kChains];
    for (int c = 0; c < kChains; ++c) x[c] = (float)(threadIdx.x + c) * 1e-3f;
    for (int i = 0; i < iters; ++i)
#pragma unroll
        for (int c = 0; c < kChains; ++c) x[c] = fmaf(x[c], a, b);
    float s = 0.f;
    for (int c = 0; c < kChains; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mb_trans(float* out, int iters) {
    float x[kChains];
    for (int c = 0; c < kChains; ++c) x[c] = (float)((threadIdx.x + c) & 7) * 0.1f;
    for (int i = 0; i < iters; ++i)
#pragma unroll
        for (int c = 0; c < kChains; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);  // stays in (0, 1]
    float s = 0.f;
    for (int c = 0; c < kChains; ++c) s += x[c];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mb_lds(uint32_t* out, int iters) {
    __shared__ __attribute__((aligned(16))) uint32_t buf[16384];  // 64 KiB
    for (int i = threadIdx.x; i < 16384; i += 256) buf[i] = i * 2654435761u;
    __syncthreads();
    u32x4 acc = {0u, 0u, 0u, 0u};
    int off = threadIdx.x * 4;  // consecutive lanes read consecutive 16-byte chunks
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(buf + ((off + c * 1024) & 16383));
            acc ^= v;
        }
        off += 4 * 256 * kChains;
    }
    out[blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

// HBM read stream: each workgroup reads its own contiguous share of the
// buffer with eight non-temporal 16-byte loads per lane in flight, each wave
// instruction covering 1 KiB of consecutive bytes -- a long sequential read
// per workgroup, as a decode workgroup streams its key and value rows.
__global__ __launch_bounds__(256) void mb_hbm(const u32x4* __restrict__ src, long long n16,
                                              uint32_t* out) {
    constexpr int U = 8;
    const long long per = (n16 + gridDim.x - 1) / gridDim.x;  // 16-byte chunks per workgroup
    const long long b0 = (long long)blockIdx.x * per;
    const long long b1 = b0 + per < n16 ? b0 + per : n16;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (long long i = b0 + threadIdx.x; i < b1; i += U * 256) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const long long j = i + u * 256;
            v[u] = j < b1 ? __builtin_nontemporal_load(src + j) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u];
    }
    out[blockIdx.x * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

template <typename F>
hipError_t time_ms(F launch, int reps, float* ms) {
    hipEvent_t a, b;
    hipError_t e = hipEventCreate(&a);
    if (e != hipSuccess) return e;
    e = hipEventCreate(&b);
    if (e != hipSuccess) return e;
    launch();  // warm up
    e = hipEventRecord(a, nullptr);
    for (int r = 0; r < reps; ++r) launch();
    if (e == hipSuccess) e = hipEventRecord(b, nullptr);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    if (e == hipSuccess) e = hipEventElapsedTime(ms, a, b);
    if (e == hipSuccess) e = hipGetLastError();
    hipEventDestroy(a);
    hipEventDestroy(b);
    if (e == hipSuccess) *ms /= reps;
    return e;
}

}  // namespace

// Runs the microbenchmarks on the current device; fills the performance
// fields of *d (structural fields must already be set).
hipError_t measure_device(attn_device_desc* d) {
    const int cus = d->num_cus;
    const double clk = d->clock_ghz * 1e9;
    const int blocks = cus * 2;  // two 4-wave workgroups per CU (compute benchmarks)
    const int hb = cus * 4;      // workgroups of the HBM stream (128 KiB in flight per CU)
    float* fout = nullptr;       // one output word per thread of the largest grid
    hipError_t e = hipMalloc(&fout, (size_t)hb * 256 * sizeof(float));
    if (e != hipSuccess) return e;
    float ms = 0.f;

    const int it_mfma = 4096;
    e = time_ms([&] { hipLaunchKernelGGL(mb_mfma, dim3(blocks), dim3(256), 0, nullptr, fout, it_mfma); },
                5, &ms);
    if (e == hipSuccess) {
        const double flops = (double)blocks * 4 * it_mfma * kChains * 32768.0;
        d->mfma_bf16_flops_per_clk_cu = flops / (ms * 1e-3) / clk / cus;
    }
    const int it_valu = 65536;
    if (e == hipSuccess)
        e = time_ms([&] { hipLaunchKernelGGL(mb_valu, dim3(blocks), dim3(256), 0, nullptr, fout, it_valu, 0.999f, 1e-3f); },
                    5, &ms);
    if (e == hipSuccess) {
        const double wave_ops = (double)blocks * 4 * it_valu * kChains;
        const double cycles_per_op = (ms * 1e-3) * clk * cus * d->simds_per_cu / wave_ops;
        d->valu_lanes_per_clk_simd = d->wave_size / cycles_per_op;
    }
    const int it_trans = 16384;
    if (e == hipSuccess)
        e = time_ms([&] { hipLaunchKernelGGL(mb_trans, dim3(blocks), dim3(256), 0, nullptr, fout, it_trans); },
                    5, &ms);
    if (e == hipSuccess) {
        const double wave_ops = (double)blocks * 4 * it_trans * kChains;
        d->trans_cycles_per_op = (ms * 1e-3) * clk * cus * d->simds_per_cu / wave_ops;
    }
    const int it_lds = 8192;
    if (e == hipSuccess)
        e = time_ms([&] { hipLaunchKernelGGL(mb_lds, dim3(blocks), dim3(256), 0, nullptr, (uint32_t*)fout, it_lds); },
                    5, &ms);
    if (e == hipSuccess) {
        const double bytes = (double)blocks * 256 * it_lds * kChains * 16.0;
        d->lds_bytes_per_clk_cu = bytes / (ms * 1e-3) / clk / cus;
    }
    if (e == hipSuccess) {
        const size_t bytes = (size_t)2 << 30;  // 2 GiB: far beyond L2 and MALL
        void* src = nullptr;
        e = hipMalloc(&src, bytes);
        if (e == hipSuccess) e = hipMemset(src, 1, bytes);
        const long long n16 = (long long)(bytes / 16);
        if (e == hipSuccess)
            e = time_ms([&] { hipLaunchKernelGGL(mb_hbm, dim3(hb), dim3(256), 0, nullptr, (const u32x4*)src, n16, (uint32_t*)fout); },
                        5, &ms);
        if (e == hipSuccess) d->hbm_bytes_per_s = (double)bytes / (ms * 1e-3);
        if (src) hipFree(src);
    }
    hipFree(fout);
    return e;
}

}  // namespace attn
