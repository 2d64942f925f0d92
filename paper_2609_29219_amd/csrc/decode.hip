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
// workspace (m in the base-2 domain).  With a single split the combine would
// be the identity (one weight 2^0 = 1), so the partial kernels then write the
// normalised output o / l, and the log-sum-exp, themselves: the same values,
// one launch less.
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

// The merged (m, l, o[c]) of row `out` (row * n_splits + split): into the
// workspace, or, with a single split (o_final set; then out is the row), as
// the final output o / l and the row's log-sum-exp (natural log).
template <int D>
__device__ __forceinline__ void store_partial(long long out, int c, float M, float L, float acc,
                                              float* ws_m, float* ws_l, float* ws_o,
                                              float* o_final, float* lse_final) {
    if (o_final) {
        o_final[out * D + c] = acc / L;
        if (lse_final && c == 0) lse_final[out] = (M + __builtin_log2f(L)) * 0.69314718055994531f;
        return;
    }
    ws_o[out * D + c] = acc;
    if (c == 0) {
        ws_m[out] = M;
        ws_l[out] = L;
    }
}

// GQ query heads that share one key/value head (grouped-query attention) run
// in the same workgroup, so each K and V row is read from memory once for
// all of them: a lane keeps GQ query slices, GQ online-softmax states and GQ
// output slices, and every loaded key is scored against each query.
template <int D, int NT, int U, int GQ>
__global__ __launch_bounds__(NT) void decode_partial_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ ws_m, float* __restrict__ ws_l,
    float* __restrict__ ws_o, float* __restrict__ o_final, float* __restrict__ lse_final, int Skv,
    int chunk, int n_splits, int group, float scale_log2) {
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
            store_partial<D>(out, c, M, L, acc, ws_m, ws_l, ws_o, o_final, lse_final);
        }
        __syncthreads();  // the LDS merge buffers are reused by the next query
    }
}

// ---------------------------------------------------------------------------
// Grouped-query decode on the matrix cores.  With G >= 4 query heads per
// key/value head, each key is scored against G queries and each value row is
// weighted G times: per key the work is a small dense product, which the
// VALU kernel above cannot keep up with at HBM speed.  Here one workgroup
// serves up to 16 query heads of one key/value head (queries padded to 16)
// over one key split, as S^T = K Q^T and O^T += V^T P^T on
// v_mfma_f32_16x16x32_bf16:
//   * Q^T (B operand: 32 dims x 16 queries) stays in registers;
//   * a wave takes 32 keys per step; K rows go from HBM straight into the A
//     operand (16 keys x 32 dims, 16 bytes per lane).  The rows are
//     permuted (block a holds keys 8g+0..3, block b keys 8g+4..7 in lane
//     group g = lane/16), so the accumulators give lane (q, g) the scores of
//     keys 8g..8g+7 of query q -- exactly the k-operand layout P^T needs;
//   * V rows are staged in the wave's own LDS tile and read transposed with
//     ds_read_b64_tr_b16 (A operand V^T: 16 dims x 32 keys);
//   * per query an online softmax (max over the four lane groups by lane
//     swaps), probabilities rounded to bf16 and the sum l over the rounded
//     values (so the output is an exact convex combination of V rows);
//   * the four waves merge through LDS and write the same unnormalised
//     (m, l, o[d]) partials per (query head, split) as the kernel above (or,
//     with a single split, the final output).
// Every memory operation is an ordinary load or LDS access the compiler
// tracks; latency is hidden by occupancy (16 KiB in flight per wave).
typedef __bf16 gq_bf16x8 __attribute__((ext_vector_type(8)));
typedef float gq_f32x4 __attribute__((ext_vector_type(4)));
typedef short gq_s16x4 __attribute__((ext_vector_type(4)));
typedef short gq_s16x8 __attribute__((ext_vector_type(8)));

// max / sum of x over the four 16-lane rows (lanes l, l^16, l^32, l^48)
__device__ __forceinline__ float rows4_max(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <int D>
__global__ __launch_bounds__(kGqaWaves * 64) void gqa_decode_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ ws_m, float* __restrict__ ws_l,
    float* __restrict__ ws_o, float* __restrict__ o_final, float* __restrict__ lse_final, int Hq,
    int Hkv, int Skv, int chunk, int n_splits, int q_blocks, int n_wg, int num_xcds,
    float scale_log2) {
    constexpr int KS = D / 32;        // MFMA k-steps over the head dimension
    constexpr int DB = D / 16;        // 16-dim blocks of O^T
    constexpr int VST = D + 32;       // bf16 per padded V row in LDS
    constexpr int VCH = 32 * D / 8;   // 16-byte chunks of a 32-key V tile
    constexpr int VI = VCH / 64;      // V chunks per lane
    static_assert(VCH % 64 == 0, "whole V tile per wave");
    __shared__ __attribute__((aligned(16))) uint16_t vtile[kGqaWaves][32 * VST];
    __shared__ float sm[kGqaWaves][16], sl[kGqaWaves][16];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, g4 = lane >> 4;

    // XCD-aware order: the query blocks of one key/value chunk are
    // neighbours in the logical order and land on one XCD (shared K/V in L2)
    const int wg = blockIdx.x;
    const int per = n_wg / num_xcds, rem = n_wg % num_xcds;
    const int xcd = wg % num_xcds, slot_id = wg / num_xcds;
    const int logical =
        (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot_id;
    const int qb = logical % q_blocks;
    const int rest = logical / q_blocks;
    const int split = rest % n_splits;
    const long long kvh = rest / n_splits;  // flat b * Hkv + h
    const int group = Hq / Hkv;
    const long long b = kvh / Hkv;
    const int q_first = (int)(kvh % Hkv) * group + qb * 16;  // first query head in batch b
    const int nq = min(16, group - qb * 16);
    const int j0 = split * chunk;
    const int j1 = min(Skv, j0 + chunk);

    // Q^T fragments: lane (q, g) holds dims 32s + 8g .. +7 of query q
    gq_bf16x8 qf[KS];
    {
        const uint16_t* qp = Q + (b * Hq + q_first + min(l16, nq - 1)) * D + 8 * g4;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            u32x4 w = *reinterpret_cast<const u32x4*>(qp + 32 * s);
            if (l16 >= nq) w = u32x4{0u, 0u, 0u, 0u};
            qf[s] = __builtin_bit_cast(gq_bf16x8, w);
        }
    }
    const uint16_t* Kb = K + kvh * (long long)Skv * D;
    const uint16_t* Vb = V + kvh * (long long)Skv * D;
    uint16_t* const vt = vtile[wave];
    const int rk = 8 * (l16 >> 2) + (l16 & 3);  // this lane's K row inside block a

    float m = -INFINITY, l = 0.f;
    gq_f32x4 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = gq_f32x4{0.f, 0.f, 0.f, 0.f};

    for (int kb = j0 + 32 * wave; kb < j1; kb += 32 * kGqaWaves) {
        // keys past the split end re-read the last key (masked to weight 0)
        u32x4 kr[2][KS], vr[VI];
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            const int key = min(kb + rk + 4 * blk, j1 - 1);
#pragma unroll
            for (int s = 0; s < KS; ++s)
                kr[blk][s] = __builtin_nontemporal_load(
                    reinterpret_cast<const u32x4*>(Kb + (long long)key * D + 32 * s + 8 * g4));
        }
#pragma unroll
        for (int i = 0; i < VI; ++i) {
            const int c = lane + 64 * i, row = c / (D / 8), cc = c % (D / 8);
            const int key = min(kb + row, j1 - 1);
            vr[i] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4*>(Vb + (long long)key * D + cc * 8));
        }
        // this wave's V tile (its earlier reads of the tile precede these
        // writes in the wave's LDS order)
#pragma unroll
        for (int i = 0; i < VI; ++i) {
            const int c = lane + 64 * i, row = c / (D / 8), cc = c % (D / 8);
            *reinterpret_cast<u32x4*>(vt + row * VST + cc * 8) = vr[i];
        }
        // scores: lane (q, g) gets keys kb + 8g + e, e = 0..7
        gq_f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(gq_bf16x8, kr[0][s]),
                                                        qf[s], sa, 0, 0, 0);
            sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(gq_bf16x8, kr[1][s]),
                                                        qf[s], sb, 0, 0, 0);
        }
        float sc[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sc[i] = sa[i];
            sc[4 + i] = sb[i];
        }
        const int room = j1 - 1 - (kb + 8 * g4);  // keys e <= room exist
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            if (e > room) sc[e] = -INFINITY;
            mx = fmaxf(mx, sc[e]);
        }
        mx = rows4_max(mx);  // key kb always exists: finite
        const float m_new = fmaxf(m, mx * scale_log2);
        const float alpha = __builtin_amdgcn_exp2f(m - m_new);
        l *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        m = m_new;
        gq_bf16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            pf[e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sc[e], scale_log2, -m));
            l += (float)pf[e];
        }
        // O^T += V^T P^T: lane (i, g) of a 16-lane group reads row 8g + i/4
        // (and + 4) at column 16 db + 4 (i % 4), and receives column
        // 16 db + i of keys 8g .. 8g+3 (and 8g+4 .. 8g+7)
        const uint16_t* vp = vt + (8 * g4 + (l16 >> 2)) * VST + 4 * (l16 & 3);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const gq_s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) gq_s16x4*)(vp + 16 * db));
            const gq_s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) gq_s16x4*)(vp + 4 * VST + 16 * db));
            const gq_s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(gq_bf16x8, w),
                                                              pf, oacc[db], 0, 0, 0);
        }
    }
    l = rows4_sum(l);  // the four lane groups summed different keys

    // merge the waves: O^T of wave w into LDS (over its V tile), then one
    // thread per (query, dim)
    __syncthreads();
    float* so = reinterpret_cast<float*>(&vtile[0][0]);  // [wave][D][16]
    static_assert(kGqaWaves * D * 16 * 4 <= (int)sizeof(vtile), "merge buffer fits");
    if (g4 == 0) {
        sm[wave][l16] = m;
        sl[wave][l16] = l;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) so[(wave * D + 16 * db + 4 * g4 + i) * 16 + l16] = oacc[db][i];
    __syncthreads();
    for (int idx = tid; idx < nq * D; idx += kGqaWaves * 64) {
        const int q = idx / D, c = idx % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kGqaWaves; ++w) M = fmaxf(M, sm[w][q]);
        float L = 0.f, acc = 0.f;
#pragma unroll
        for (int w = 0; w < kGqaWaves; ++w) {
            const float wt = __builtin_amdgcn_exp2f(sm[w][q] - M);  // waves without keys: 0
            L = fmaf(wt, sl[w][q], L);
            acc = fmaf(wt, so[(w * D + c) * 16 + q], acc);
        }
        const long long out = (b * Hq + q_first + q) * n_splits + split;
        store_partial<D>(out, c, M, L, acc, ws_m, ws_l, ws_o, o_final, lse_final);
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
                                 float* o_final, float* lse_final, long long BHq, int Skv,
                                 int group, float scale_log2, hipStream_t st) {
    // fewer keys in flight per lane group when each key serves many queries
    constexpr int U = GQ >= 4 ? 4 : kDecodeUnroll;
    hipLaunchKernelGGL((decode_partial_kernel<D, kDecodeThreads, U, GQ>),
                       dim3((unsigned)(BHq / GQ * p.n_splits)), dim3(kDecodeThreads), 0, st,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                       static_cast<const uint16_t*>(v), ws_m, ws_l, ws_o, o_final, lse_final,
                       Skv, p.chunk, p.n_splits, group, scale_log2);
    return hipGetLastError();
}

template <int D>
static hipError_t launch_decode_d(const DecodePlan& p, const void* q, const void* k,
                                  const void* v, float* o, float* lse, float* ws, int B, int Hq,
                                  int Hkv, int Skv, float scale_log2, int num_xcds,
                                  hipStream_t st) {
    const long long BHq = (long long)B * Hq;
    const int group = Hq / Hkv;
    float* ws_m = ws;
    float* ws_l = ws + BHq * p.n_splits;
    float* ws_o = ws + 2 * BHq * p.n_splits;
    // a single split writes the output directly (no combine launch)
    const bool direct = p.n_splits == 1;
    float* const o_final = direct ? o : nullptr;
    float* const lse_final = direct ? lse : nullptr;
    hipError_t e = hipErrorInvalidValue;
    if (p.mfma) {
        if (p.grid > 0x7fffffffLL || p.q_blocks != (group + 15) / 16) return hipErrorInvalidValue;
        hipLaunchKernelGGL((gqa_decode_kernel<D>), dim3((unsigned)p.grid), dim3(kGqaWaves * 64), 0,
                           st, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                           static_cast<const uint16_t*>(v), ws_m, ws_l, ws_o, o_final, lse_final,
                           Hq, Hkv, Skv, p.chunk, p.n_splits, p.q_blocks, (int)p.grid, num_xcds,
                           scale_log2);
        e = hipGetLastError();
        if (e != hipSuccess || direct) return e;
        return launch_split_combine(D, ws_m, ws_l, ws_o, o, 0, lse, BHq, p.n_splits, st);
    }
    switch (decode_heads_per_wg(group)) {
        case 8: e = launch_partial<D, 8>(p, q, k, v, ws_m, ws_l, ws_o, o_final, lse_final, BHq, Skv, group, scale_log2, st); break;
        case 4: e = launch_partial<D, 4>(p, q, k, v, ws_m, ws_l, ws_o, o_final, lse_final, BHq, Skv, group, scale_log2, st); break;
        case 2: e = launch_partial<D, 2>(p, q, k, v, ws_m, ws_l, ws_o, o_final, lse_final, BHq, Skv, group, scale_log2, st); break;
        default: e = launch_partial<D, 1>(p, q, k, v, ws_m, ws_l, ws_o, o_final, lse_final, BHq, Skv, group, scale_log2, st);
    }
    if (e != hipSuccess || direct) return e;
    return launch_split_combine(D, ws_m, ws_l, ws_o, o, 0, lse, BHq, p.n_splits, st);
}

hipError_t launch_decode(const DecodePlan& p, const void* q, const void* k, const void* v,
                         float* o, float* lse, float* workspace, int B, int Hq, int Hkv, int Skv,
                         float scale, int num_xcds, hipStream_t stream) {
    const float scale_log2 = (float)((double)scale * 1.4426950408889634);
    if (p.d == 64)
        return launch_decode_d<64>(p, q, k, v, o, lse, workspace, B, Hq, Hkv, Skv, scale_log2,
                                   num_xcds, stream);
    if (p.d == 128)
        return launch_decode_d<128>(p, q, k, v, o, lse, workspace, B, Hq, Hkv, Skv, scale_log2,
                                    num_xcds, stream);
    return hipErrorInvalidValue;
}

}  // namespace attn
