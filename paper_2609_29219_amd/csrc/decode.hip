// Flash-Decode for gfx950: one query per (batch, head), the key sequence split
// into chunks processed by separate workgroups, then a combine kernel.
//
// The split follows the paper's Flash Decode decomposition (HEG paragraph
// of the latency-modelling section): a local softmax loop per chunk, a
// gather of the partial results, a global softmax over them and the final
// output.  Here the local loop is decode_partial_kernel and the gather +
// global softmax + final output is decode_combine_kernel.
//
// decode_partial_kernel.  The work is a stream over K and V (HBM bound: 4*d
// bytes per key against 4*d flops).  G = d/8 lanes share one key: each lane
// loads 16 contiguous bytes of the key's K row and of its V row, so a wave
// load instruction covers 64/G whole rows (1 KiB contiguous).  Each lane
// group keeps its own online-softmax state (max m, sum l, 8 output dims per
// lane); a step handles U keys per group, all loads of a step issued before
// any use.  The q.k dot product is reduced across the G lanes with DPP.
// At the end the groups of the workgroup merge through LDS, and the
// workgroup writes (m, l, o[d]) of its split, unnormalised, to the
// workspace (m in the base-2 domain).
#include "common.h"

namespace attn {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Sum over the G consecutive lanes of a group (G = 8 or 16), result in every
// lane of the group.  quad_perm[1,0,3,2], quad_perm[2,3,0,1], then
// row_half_mirror (lane i <- 7-i inside 8) and row_mirror (i <- 15-i inside 16).
template <int G>
__device__ __forceinline__ float group_sum(float x) {
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));
    if (G == 16)
        x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, false));
    return x;
}

template <int D, int NT, int U>
__global__ __launch_bounds__(NT) void decode_partial_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ ws_m, float* __restrict__ ws_l,
    float* __restrict__ ws_o, int Skv, int chunk, int n_splits, float scale_log2) {
    constexpr int G = D / 8;      // lanes per key
    constexpr int NG = NT / G;    // lane groups (keys per step) in the workgroup
    const int tid = threadIdx.x;
    const int gid = tid / G, sub = tid % G;
    const int split = blockIdx.x % n_splits;
    const long long bh = blockIdx.x / n_splits;
    const int j0 = split * chunk;
    const int j1 = min(Skv, j0 + chunk);

    // this lane's 8 query dims, pre-multiplied by scale*log2(e)
    float qv[8];
    {
        const u32x4 w = *reinterpret_cast<const u32x4*>(Q + bh * D + sub * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            qv[2 * e] = __uint_as_float(w[e] << 16) * scale_log2;
            qv[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u) * scale_log2;
        }
    }

    const uint16_t* Kb = K + bh * (long long)Skv * D + sub * 8;
    const uint16_t* Vb = V + bh * (long long)Skv * D + sub * 8;

    float m = -INFINITY, l = 0.f;
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.f;

    for (int base = j0; base < j1; base += U * NG) {
        u32x4 kr[U], vr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            // keys past the split end reuse the last valid row (weight 0)
            const int key = min(base + u * NG + gid, j1 - 1);
            kr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Kb + (long long)key * D));
            vr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Vb + (long long)key * D));
        }
        float s[U];
        float mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            float acc = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc = fmaf(qv[2 * e], __uint_as_float(kr[u][e] << 16), acc);
                acc = fmaf(qv[2 * e + 1], __uint_as_float(kr[u][e] & 0xffff0000u), acc);
            }
            acc = group_sum<G>(acc);
            s[u] = (base + u * NG + gid < j1) ? acc : -INFINITY;
            mx = fmaxf(mx, s[u]);
        }
        const float m_new = fmaxf(m, mx);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m - m_use);
        l *= alpha;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] *= alpha;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float p = __builtin_amdgcn_exp2f(s[u] - m_use);
            l += p;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                o[2 * e] = fmaf(p, __uint_as_float(vr[u][e] << 16), o[2 * e]);
                o[2 * e + 1] = fmaf(p, __uint_as_float(vr[u][e] & 0xffff0000u), o[2 * e + 1]);
            }
        }
        m = m_new;
    }

    // merge the NG lane groups of this workgroup
    __shared__ float sm[NG], sl[NG];
    __shared__ float so[NG][D + 4];
    if (sub == 0) {
        sm[gid] = m;
        sl[gid] = l;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) so[gid][sub * 8 + e] = o[e];
    __syncthreads();
    const long long out = bh * n_splits + split;
    for (int c = tid; c < D; c += NT) {
        float M = -INFINITY;
        for (int g = 0; g < NG; ++g) M = fmaxf(M, sm[g]);
        float L = 0.f, acc = 0.f;
        for (int g = 0; g < NG; ++g) {
            const float w = __builtin_amdgcn_exp2f(sm[g] - M);
            L = fmaf(w, sl[g], L);
            acc = fmaf(w, so[g][c], acc);
        }
        ws_o[out * D + c] = acc;
        if (c == 0) {
            ws_m[out] = M;
            ws_l[out] = L;
        }
    }
}

// Global softmax over the split partials and the final output:
//   M = max_s m_s, w_s = 2^(m_s - M), o = sum_s w_s o_s / sum_s w_s l_s.
template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(const float* __restrict__ ws_m,
                                                           const float* __restrict__ ws_l,
                                                           const float* __restrict__ ws_o,
                                                           float* __restrict__ O, int n_splits) {
    const long long bh = blockIdx.x;
    const int c = threadIdx.x;
    const float* mm = ws_m + bh * n_splits;
    const float* ll = ws_l + bh * n_splits;
    const float* oo = ws_o + bh * n_splits * D + c;
    float M = -INFINITY;
    for (int s = 0; s < n_splits; ++s) M = fmaxf(M, mm[s]);
    float L = 0.f, acc = 0.f;
    for (int s = 0; s < n_splits; ++s) {
        const float w = __builtin_amdgcn_exp2f(mm[s] - M);
        L = fmaf(w, ll[s], L);
        acc = fmaf(w, oo[(long long)s * D], acc);
    }
    O[bh * D + c] = acc / L;
}

template <int D>
static hipError_t launch_decode_d(const DecodePlan& p, const void* q, const void* k,
                                  const void* v, float* o, float* ws, int B, int H, int Skv,
                                  float scale_log2, hipStream_t st) {
    const long long BH = (long long)B * H;
    float* ws_m = ws;
    float* ws_l = ws + BH * p.n_splits;
    float* ws_o = ws + 2 * BH * p.n_splits;
    hipLaunchKernelGGL((decode_partial_kernel<D, kDecodeThreads, kDecodeUnroll>),
                       dim3((unsigned)(BH * p.n_splits)), dim3(kDecodeThreads), 0, st,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), ws_m, ws_l, ws_o, Skv, p.chunk,
                       p.n_splits, scale_log2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_combine_kernel<D>), dim3((unsigned)BH), dim3(D), 0, st, ws_m, ws_l,
                       ws_o, o, p.n_splits);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodePlan& p, const void* q, const void* k, const void* v,
                         float* o, float* workspace, int B, int H, int Skv, float scale,
                         hipStream_t stream) {
    const float scale_log2 = (float)((double)scale * 1.4426950408889634);
    if (p.d == 64) return launch_decode_d<64>(p, q, k, v, o, workspace, B, H, Skv, scale_log2, stream);
    if (p.d == 128) return launch_decode_d<128>(p, q, k, v, o, workspace, B, H, Skv, scale_log2, stream);
    return hipErrorInvalidValue;
}

}  // namespace attn
