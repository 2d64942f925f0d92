// A caller of libattn.so's C ABI with nothing but the HIP runtime: no Python,
// no torch in the process.  It allocates device buffers itself, runs the
// prefill and decode entry points on inputs whose results have closed forms,
// checks them, and checks that an unsupported call fails with a message.
//
// Closed forms (softmax attention as the paper states it, Evaluation,
// Experimental Setup):
//   - every V row equal to r: the weights sum to one, so O = r;
//   - Q = 0: every allowed key has weight 1 / (number of allowed keys), so O
//     is the mean of the allowed V rows (all rows; the prefix for causal rows);
//   - decode with Q = 0: the mean of all V rows of the head.
// Prints "abi_check ok" and exits 0 when every check holds.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "attn.h"

namespace {

int g_failures = 0;

void expect(bool ok, const char* what) {
    if (!ok) {
        std::fprintf(stderr, "FAILED: %s\n", what);
        ++g_failures;
    }
}

#define HIP_OK(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess) {                                                       \
            std::fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));           \
            std::exit(2);                                                             \
        }                                                                             \
    } while (0)

// bf16 by round-to-nearest-even of an fp32 value (inputs are finite)
uint16_t to_bf16(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

float from_bf16(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}

// deterministic values in [-2, 2): a 64-bit LCG, top bits
struct Lcg {
    uint64_t s;
    float next() {
        s = s * 6364136223846793005ull + 1442695040888963407ull;
        return (float)((s >> 40) & 0xffffff) / (float)(1 << 24) * 4.f - 2.f;
    }
};

template <typename T>
T* device_copy(const std::vector<T>& h) {
    T* d = nullptr;
    HIP_OK(hipMalloc(&d, h.size() * sizeof(T)));
    HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
    return d;
}

template <typename T>
std::vector<T> host_copy(const T* d, size_t n) {
    std::vector<T> h(n);
    HIP_OK(hipMemcpy(h.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
    return h;
}

double max_rel_err(const std::vector<float>& got, const std::vector<double>& want) {
    double worst = 0;
    for (size_t i = 0; i < got.size(); ++i) {
        const double e = std::fabs(got[i] - want[i]) / std::fmax(1.0, std::fabs(want[i]));
        worst = std::fmax(worst, std::isfinite(got[i]) ? e : INFINITY);
    }
    return worst;
}

// prefill: identical V rows, then Q = 0 (full and causal)
void check_prefill(int B, int H, int Sq, int Skv, int d) {
    const size_t nq = (size_t)B * H * Sq * d, nkv = (size_t)B * H * Skv * d;
    Lcg g{(uint64_t)(B * 131 + H * 17 + Sq * 7 + Skv + d)};
    std::vector<uint16_t> q(nq), k(nkv), v(nkv);
    for (auto& x : q) x = to_bf16(g.next());
    for (auto& x : k) x = to_bf16(g.next());
    // V: every key of a head holds the same row r_h
    std::vector<double> want_same(nq);
    for (int bh = 0; bh < B * H; ++bh) {
        std::vector<uint16_t> r(d);
        for (auto& x : r) x = to_bf16(g.next());
        for (int j = 0; j < Skv; ++j)
            std::memcpy(&v[((size_t)bh * Skv + j) * d], r.data(), d * 2);
        for (int i = 0; i < Sq; ++i)
            for (int c = 0; c < d; ++c) want_same[((size_t)bh * Sq + i) * d + c] = from_bf16(r[c]);
    }
    uint16_t *dq = device_copy(q), *dk = device_copy(k), *dv = device_copy(v);
    float* dout = nullptr;
    HIP_OK(hipMalloc(&dout, nq * sizeof(float)));
    const float scale = 1.0f / std::sqrt((float)d);
    for (int causal = 0; causal < 2; ++causal) {
        expect(attn_fwd(dq, dk, dv, dout, B, H, Sq, Skv, d, scale, causal) == ATTN_OK,
               "attn_fwd (identical V rows) returns ATTN_OK");
        HIP_OK(hipDeviceSynchronize());
        expect(max_rel_err(host_copy(dout, nq), want_same) <= 1e-5,
               "attn_fwd with identical V rows gives that row");
    }
    // Q = 0 with varied V: the mean of the allowed rows
    for (auto& x : v) x = to_bf16(g.next());
    HIP_OK(hipMemcpy(dv, v.data(), nkv * 2, hipMemcpyHostToDevice));
    HIP_OK(hipMemset(dq, 0, nq * 2));
    for (int causal = 0; causal < 2; ++causal) {
        std::vector<double> want(nq);
        for (int bh = 0; bh < B * H; ++bh)
            for (int i = 0; i < Sq; ++i) {
                const int allowed = causal ? i + (Skv - Sq) + 1 : Skv;
                for (int c = 0; c < d; ++c) {
                    double s = 0;
                    for (int j = 0; j < allowed; ++j)
                        s += from_bf16(v[((size_t)bh * Skv + j) * d + c]);
                    want[((size_t)bh * Sq + i) * d + c] = s / allowed;
                }
            }
        expect(attn_fwd(dq, dk, dv, dout, B, H, Sq, Skv, d, scale, causal) == ATTN_OK,
               "attn_fwd (Q = 0) returns ATTN_OK");
        HIP_OK(hipDeviceSynchronize());
        expect(max_rel_err(host_copy(dout, nq), want) <= 1e-4,
               causal ? "causal attn_fwd with Q = 0 gives the prefix mean of V"
                      : "attn_fwd with Q = 0 gives the mean of V");
    }
    HIP_OK(hipFree(dq));
    HIP_OK(hipFree(dk));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(dout));
}

// decode with Q = 0 for several split counts: the mean of the head's V rows
void check_decode(int B, int H, int Skv, int d) {
    const size_t nq = (size_t)B * H * d, nkv = (size_t)B * H * Skv * d;
    Lcg g{(uint64_t)(B * 7 + H * 3 + Skv + d)};
    std::vector<uint16_t> q(nq, 0), k(nkv), v(nkv);
    for (auto& x : k) x = to_bf16(g.next());
    for (auto& x : v) x = to_bf16(g.next());
    std::vector<double> want(nq);
    for (int bh = 0; bh < B * H; ++bh)
        for (int c = 0; c < d; ++c) {
            double s = 0;
            for (int j = 0; j < Skv; ++j) s += from_bf16(v[((size_t)bh * Skv + j) * d + c]);
            want[(size_t)bh * d + c] = s / Skv;
        }
    uint16_t *dq = device_copy(q), *dk = device_copy(k), *dv = device_copy(v);
    float* dout = nullptr;
    HIP_OK(hipMalloc(&dout, nq * sizeof(float)));
    for (int n : {0, 1, 5, 32}) {
        expect(attn_decode(dq, dk, dv, dout, B, H, Skv, d, n) == ATTN_OK,
               "attn_decode returns ATTN_OK");
        HIP_OK(hipDeviceSynchronize());
        expect(max_rel_err(host_copy(dout, nq), want) <= 1e-4,
               "attn_decode with Q = 0 gives the mean of V");
    }
    HIP_OK(hipFree(dq));
    HIP_OK(hipFree(dk));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(dout));
}

}  // namespace

int main() {
    attn_device_desc desc;
    expect(attn_query_device(&desc) == ATTN_OK, "attn_query_device finds the device");
    std::printf("device %s, %d CUs\n", desc.arch, desc.num_cus);
    check_prefill(2, 3, 100, 300, 64);
    check_prefill(1, 2, 257, 257, 128);
    check_decode(2, 4, 1500, 128);
    check_decode(1, 3, 77, 64);
    // an unsupported head dimension is refused on the host, with a message
    uint16_t* dummy = nullptr;
    HIP_OK(hipMalloc(&dummy, 4096));
    expect(attn_fwd(dummy, dummy, dummy, (float*)dummy, 1, 1, 4, 4, 96, 0.1f, 0) ==
               ATTN_EUNSUPPORTED,
           "head dim 96 is ATTN_EUNSUPPORTED");
    expect(std::strlen(attn_last_error()) > 0, "attn_last_error explains the refusal");
    HIP_OK(hipFree(dummy));
    if (g_failures) {
        std::fprintf(stderr, "abi_check: %d check(s) failed\n", g_failures);
        return 1;
    }
    std::printf("abi_check ok\n");
    return 0;
}
