// Flash-Decode for gfx950: one query per (batch, head), the key sequence split
// into chunks processed by separate workgroups, then a combine kernel.
//
// The split follows the paper's Flash Decode decomposition (HEG paragraph
// of the latency-modelling section): a local softmax loop per chunk, a
// gather of the partial results, a global softmax over them and the final
// output.  Here the local loop is decode_partial_kernel and the gather +
// global softmax + final output is split_combine_kernel.
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

// GQ query heads that share one key/value head (grouped-query attention) run
// in the same workgroup, so each K and V row is read from memory once for
// all of them: a lane keeps GQ query slices, GQ online-softmax states and GQ
// output slices, and every loaded key is scored against each query.
template <int D, int NT, int U, int GQ>
__global__ __launch_bounds__(NT) void decode_partial_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ ws_m, float* __restrict__ ws_l,
    float* __restrict__ ws_o, int Skv, int chunk, int n_splits, int group, float scale_log2) {
    constexpr int G = D / 8;      // lanes per key
    constexpr int NG = NT / G;    // lane groups (keys per step) in the workgroup
    const int tid = threadIdx.x;
    const int gid = tid / G, sub = tid % G;
    const int split = blockIdx.x % n_splits;
    // blockIdx / n_splits enumerates (b, query-head block of GQ heads)
    const long long hb = blockIdx.x / n_splits;
    const long long bh0 = hb * GQ;          // first query head (flat b*Hq + h)
    const long long kvh = bh0 / group;      // the key/value head they share
    const int j0 = split * chunk;
    const int j1 = min(Skv, j0 + chunk);

    // this lane's 8 dims of each query, pre-multiplied by scale*log2(e)
    float qv[GQ][8];
#pragma unroll
    for (int g = 0; g < GQ; ++g) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(Q + (bh0 + g) * D + sub * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            qv[g][2 * e] = __uint_as_float(w[e] << 16) * scale_log2;
            qv[g][2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u) * scale_log2;
        }
    }

    const uint16_t* Kb = K + kvh * (long long)Skv * D + sub * 8;
    const uint16_t* Vb = V + kvh * (long long)Skv * D + sub * 8;

    float m[GQ], l[GQ], o[GQ][8];
#pragma unroll
    for (int g = 0; g < GQ; ++g) {
        m[g] = -INFINITY;
        l[g] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[g][e] = 0.f;
    }

    for (int base = j0; base < j1; base += U * NG) {
        u32x4 kr[U], vr[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            // keys past the split end reuse the last valid row (weight 0)
            const int key = min(base + u * NG + gid, j1 - 1);
            kr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Kb + (long long)key * D));
            vr[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Vb + (long long)key * D));
        }
#pragma unroll
        for (int g = 0; g < GQ; ++g) {
            float s[U];
            float mx = -INFINITY;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc = fmaf(qv[g][2 * e], __uint_as_float(kr[u][e] << 16), acc);
                    acc = fmaf(qv[g][2 * e + 1], __uint_as_float(kr[u][e] & 0xffff0000u), acc);
                }
                acc = group_sum<G>(acc);
                s[u] = (base + u * NG + gid < j1) ? acc : -INFINITY;
                mx = fmaxf(mx, s[u]);
            }
            const float m_new = fmaxf(m[g], mx);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            const float alpha = __builtin_amdgcn_exp2f(m[g] - m_use);
            l[g] *= alpha;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[g][e] *= alpha;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float p = __builtin_amdgcn_exp2f(s[u] - m_use);
                l[g] += p;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    o[g][2 * e] = fmaf(p, __uint_as_float(vr[u][e] << 16), o[g][2 * e]);
                    o[g][2 * e + 1] =
                        fmaf(p, __uint_as_float(vr[u][e] & 0xffff0000u), o[g][2 * e + 1]);
                }
            }
            m[g] = m_new;
        }
    }

    // merge the NG lane groups of this workgroup, one query at a time
    __shared__ float sm[NG], sl[NG];
    __shared__ float so[NG][D + 4];
#pragma unroll
    for (int g = 0; g < GQ; ++g) {
        if (sub == 0) {
            sm[gid] = m[g];
            sl[gid] = l[g];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) so[gid][sub * 8 + e] = o[g][e];
        __syncthreads();
        const long long out = (bh0 + g) * n_splits + split;
        for (int c = tid; c < D; c += NT) {
            float M = -INFINITY;
            for (int q = 0; q < NG; ++q) M = fmaxf(M, sm[q]);
            float L = 0.f, acc = 0.f;
            for (int q = 0; q < NG; ++q) {
                const float w = __builtin_amdgcn_exp2f(sm[q] - M);
                L = fmaf(w, sl[q], L);
                acc = fmaf(w, so[q][c], acc);
            }
            ws_o[out * D + c] = acc;
            if (c == 0) {
                ws_m[out] = M;
                ws_l[out] = L;
            }
        }
        __syncthreads();  // the LDS merge buffers are reused by the next query
    }
}

// Global softmax over the split partials and the final output:
//   M = max_s m_s, w_s = 2^(m_s - M), o = sum_s w_s o_s / sum_s w_s l_s,
// and optionally the log-sum-exp of the row's scores (natural log),
//   lse = (M + log2(sum_s w_s l_s)) * ln 2.
// One workgroup of D threads per row; the partials of row r are at r*n + s.
// Used by decode and by split-key prefill (fp32 or bf16 output).
template <int D>
__global__ __launch_bounds__(D) void split_combine_kernel(const float* __restrict__ ws_m,
                                                          const float* __restrict__ ws_l,
                                                          const float* __restrict__ ws_o,
                                                          void* __restrict__ O, int out_bf16,
                                                          float* __restrict__ lse, int n_splits) {
    const long long r = blockIdx.x;
    const int c = threadIdx.x;
    const float* mm = ws_m + r * n_splits;
    const float* ll = ws_l + r * n_splits;
    const float* oo = ws_o + r * n_splits * D + c;
    float M = -INFINITY;
    for (int s = 0; s < n_splits; ++s) M = fmaxf(M, mm[s]);
    float L = 0.f, acc = 0.f;
    for (int s = 0; s < n_splits; ++s) {
        const float w = __builtin_amdgcn_exp2f(mm[s] - M);
        L = fmaf(w, ll[s], L);
        acc = fmaf(w, oo[(long long)s * D], acc);
    }
    const float val = acc / L;
    if (out_bf16)
        static_cast<__bf16*>(O)[r * D + c] = (__bf16)val;
    else
        static_cast<float*>(O)[r * D + c] = val;
    if (lse && c == 0) lse[r] = (M + __builtin_log2f(L)) * 0.69314718055994531f;
}

hipError_t launch_split_combine(int d, const float* ws_m, const float* ws_l, const float* ws_o,
                                void* o, int out_bf16, float* lse, long long rows, int n_splits,
                                hipStream_t st) {
    // one workgroup of d threads per row; a grid holds at most 2^32 - 1 threads
    if (rows <= 0 || rows * d > 0xffffffffLL) return hipErrorInvalidValue;
    if (d == 64)
        hipLaunchKernelGGL((split_combine_kernel<64>), dim3((unsigned)rows), dim3(64), 0, st,
                           ws_m, ws_l, ws_o, o, out_bf16, lse, n_splits);
    else if (d == 128)
        hipLaunchKernelGGL((split_combine_kernel<128>), dim3((unsigned)rows), dim3(128), 0, st,
                           ws_m, ws_l, ws_o, o, out_bf16, lse, n_splits);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int D, int GQ>
static hipError_t launch_partial(const DecodePlan& p, const void* q, const void* k,
                                 const void* v, float* ws_m, float* ws_l, float* ws_o,
                                 long long BHq, int Skv, int group, float scale_log2,
                                 hipStream_t st) {
    // fewer keys in flight per lane group when each key serves many queries
    constexpr int U = GQ >= 4 ? 4 : kDecodeUnroll;
    hipLaunchKernelGGL((decode_partial_kernel<D, kDecodeThreads, U, GQ>),
                       dim3((unsigned)(BHq / GQ * p.n_splits)), dim3(kDecodeThreads), 0, st,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), ws_m, ws_l, ws_o, Skv, p.chunk,
                       p.n_splits, group, scale_log2);
    return hipGetLastError();
}

template <int D>
static hipError_t launch_decode_d(const DecodePlan& p, const void* q, const void* k,
                                  const void* v, float* o, float* lse, float* ws, int B, int Hq,
                                  int Hkv, int Skv, float scale_log2, hipStream_t st) {
    const long long BHq = (long long)B * Hq;
    const int group = Hq / Hkv;
    float* ws_m = ws;
    float* ws_l = ws + BHq * p.n_splits;
    float* ws_o = ws + 2 * BHq * p.n_splits;
    hipError_t e = hipErrorInvalidValue;
    switch (decode_heads_per_wg(group)) {
        case 8: e = launch_partial<D, 8>(p, q, k, v, ws_m, ws_l, ws_o, BHq, Skv, group, scale_log2, st); break;
        case 4: e = launch_partial<D, 4>(p, q, k, v, ws_m, ws_l, ws_o, BHq, Skv, group, scale_log2, st); break;
        case 2: e = launch_partial<D, 2>(p, q, k, v, ws_m, ws_l, ws_o, BHq, Skv, group, scale_log2, st); break;
        default: e = launch_partial<D, 1>(p, q, k, v, ws_m, ws_l, ws_o, BHq, Skv, group, scale_log2, st);
    }
    if (e != hipSuccess) return e;
    return launch_split_combine(D, ws_m, ws_l, ws_o, o, 0, lse, BHq, p.n_splits, st);
}

hipError_t launch_decode(const DecodePlan& p, const void* q, const void* k, const void* v,
                         float* o, float* lse, float* workspace, int B, int Hq, int Hkv, int Skv,
                         float scale, hipStream_t stream) {
    const float scale_log2 = (float)((double)scale * 1.4426950408889634);
    if (p.d == 64)
        return launch_decode_d<64>(p, q, k, v, o, lse, workspace, B, Hq, Hkv, Skv, scale_log2, stream);
    if (p.d == 128)
        return launch_decode_d<128>(p, q, k, v, o, lse, workspace, B, Hq, Hkv, Skv, scale_log2, stream);
    return hipErrorInvalidValue;
}

}  // namespace attn
