// Prefill attention kernel for gfx950 (CDNA4).
//
// One workgroup computes BLOCK_M = 32*NW query rows of one (batch, head)
// against all allowed keys, streaming K/V in tiles of BN keys through LDS
// with an online softmax (running max m, running sum l, rescaled output).
//
// Operand orientation.  Each wave owns 32 query rows and computes the
// transposed score block S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// (A = 32 keys x 16 dims from LDS, B = 16 dims x 32 queries held in VGPRs).
// The 32x32 accumulator puts one query column in each lane (lane & 31) and
// 16 keys of it in that lane's 16 registers (the other 16 keys sit in lane
// ^ 32).  The row max and row sum are therefore in-lane reductions plus one
// exchange between the two wave halves.
//
// Key permutation.  Accumulator register r of lane half h holds MFMA row
// 8*(r/4) + 4*h + r%4.  K rows are written to LDS permuted inside each
// 32-key block (LDS row p holds key 16*((p%8)/4) + 4*(p/8) + p%4), so
// register r of half h is key 16*h + r: a lane's 16 probabilities are 16
// consecutive keys, which is exactly the k-operand layout the PV MFMA needs.
//
// PV.  O^T += V^T P^T with A = V^T (32 dims x 16 keys) read from a
// transposed V tile in LDS and B = the bf16 probabilities straight from
// registers.  The output accumulator again has one query per lane, so the
// online-softmax rescale is one per-lane scalar.
//
// Pipelining (the HEG pipe knob on the load/body boundary): DBUF = 1 keeps
// two LDS slots and issues the global loads of tile t+1 before computing
// tile t; DBUF = 0 loads, waits and computes in sequence.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int D, int BN>
struct FwdLds {
    static constexpr int K_STRIDE = D + 8;   // bf16 per K row (16-byte pad)
    static constexpr int V_STRIDE = BN + 8;  // bf16 per V^T row (16-byte pad)
    static constexpr int K_ELEMS = BN * K_STRIDE;
    static constexpr int V_ELEMS = D * V_STRIDE;
    static constexpr int SLOT = K_ELEMS + V_ELEMS;
};

// LDS row of key j (0..31) inside a 32-key block; inverse of the permutation
// described above.
__device__ __forceinline__ int k_lds_row(int j) {
    return ((j >> 2) & 3) << 3 | (j >> 4) << 2 | (j & 3);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Waves per SIMD the register allocator should leave room for: two when two
// workgroups' LDS fits in one CU (or one 8-wave workgroup), else one.
template <int D, int BN, int NW, bool DBUF>
constexpr int fwd_waves_per_eu() {
    constexpr int lds = (DBUF ? 2 : 1) * FwdLds<D, BN>::SLOT * 2;
    constexpr int wgs = 163840 / lds;
    return (wgs * NW / 4) >= 2 ? 2 : 1;
}

template <int D, int BN, int NW, bool DBUF, bool CAUSAL>
__global__ __launch_bounds__(NW * 64, (fwd_waves_per_eu<D, BN, NW, DBUF>())) void fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ O, int Sq, int Skv, int n_qtiles,
    int n_wg, int num_xcds, float scale_log2, uint32_t q_sign) {
    constexpr int BM = NW * 32;
    constexpr int NT = NW * 64;
    constexpr int KD = D / 16;   // MFMA k-steps over the head dimension
    constexpr int KB = BN / 32;  // 32-key blocks per tile
    constexpr int CB = D / 32;   // 32-dim blocks of the output
    using L = FwdLds<D, BN>;
    constexpr int K_CHUNKS = BN * D / 8;         // 16-byte chunks of a K tile
    constexpr int V_GROUPS = (BN / 4) * (D / 8); // 4 keys x 8 dims groups of V
    constexpr int KCH = (K_CHUNKS + NT - 1) / NT;
    constexpr int VCH = (V_GROUPS + NT - 1) / NT;

    __shared__ __attribute__((aligned(16))) uint16_t lds[(DBUF ? 2 : 1) * L::SLOT];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int l32 = lane & 31;
    const int hh = lane >> 5;

    // XCD-aware workgroup order: the hardware deals workgroup ids round-robin
    // to the XCDs, so give each XCD a contiguous range of logical tiles (the
    // q-tiles of a few heads), whose K/V then stay in that XCD's L2.
    const int wg = blockIdx.x;
    const int per = n_wg / num_xcds, rem = n_wg % num_xcds;
    const int xcd = wg % num_xcds, slot_id = wg / num_xcds;
    const int logical =
        (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot_id;
    const int bh = logical / n_qtiles;
    const int qt_order = logical % n_qtiles;
    // causal: heaviest q-tiles (most keys) first within each head
    const int qt = CAUSAL ? (n_qtiles - 1 - qt_order) : qt_order;

    const int q_wave0 = qt * BM + wave * 32;  // first query row of this wave
    const int qrow = q_wave0 + l32;
    const int diag = Skv - Sq;                // causal: key j allowed iff j <= row + diag

    // ---- Q tile into VGPRs, as the B operand (16 dims x 32 queries) --------
    bf16x8 qf[KD];
    {
        const uint16_t* qp = Q + ((long long)bh * Sq + qrow) * D + hh * 8;
#pragma unroll
        for (int ks = 0; ks < KD; ++ks) {
            u32x4 w = {0u, 0u, 0u, 0u};
            if (qrow < Sq) w = *reinterpret_cast<const u32x4*>(qp + ks * 16);
            w ^= q_sign;  // exact negation for a negative scale
            qf[ks] = __builtin_bit_cast(bf16x8, w);
        }
    }

    // ---- key range of this workgroup ------------------------------------
    int kv_end = Skv;
    if (CAUSAL) {
        const int last_q = min(qt * BM + BM - 1, Sq - 1);
        kv_end = min(Skv, last_q + diag + 1);
    }
    const int n_tiles = (kv_end + BN - 1) / BN;

    const long long kv_base = (long long)bh * Skv * D;
    const uint16_t* Kb = K + kv_base;
    const uint16_t* Vb = V + kv_base;

    u32x4 kreg[KCH];
    u32x4 vreg[VCH][4];

    auto load_tile = [&](int t) {
        const int key0 = t * BN;
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const int u = tid + i * NT;
            kreg[i] = u32x4{0u, 0u, 0u, 0u};
            if (u < K_CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                if (key0 + j < Skv)
                    kreg[i] = *reinterpret_cast<const u32x4*>(Kb + (long long)(key0 + j) * D + cc * 8);
            }
        }
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            const int g = tid + i * NT;
#pragma unroll
            for (int r = 0; r < 4; ++r) vreg[i][r] = u32x4{0u, 0u, 0u, 0u};
            if (g < V_GROUPS) {
                const int kq = g / (D / 8), cc = g % (D / 8);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int key = key0 + 4 * kq + r;
                    if (key < Skv)
                        vreg[i][r] = *reinterpret_cast<const u32x4*>(Vb + (long long)key * D + cc * 8);
                }
            }
        }
    };

    auto store_tile = [&](uint16_t* slot) {
        uint16_t* kl = slot;
        uint16_t* vl = slot + L::K_ELEMS;
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const int u = tid + i * NT;
            if (u < K_CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                const int prow = (j & ~31) | k_lds_row(j & 31);
                *reinterpret_cast<u32x4*>(kl + prow * L::K_STRIDE + cc * 8) = kreg[i];
            }
        }
        // V is written transposed: V^T[dim][key], 4 keys (8 bytes) per store.
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            const int g = tid + i * NT;
            if (g < V_GROUPS) {
                const int kq = g / (D / 8), cc = g % (D / 8);
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const uint32_t a0 = vreg[i][0][w], a1 = vreg[i][1][w];
                    const uint32_t a2 = vreg[i][2][w], a3 = vreg[i][3][w];
                    u32x2 even = {(a0 & 0xffffu) | (a1 << 16), (a2 & 0xffffu) | (a3 << 16)};
                    u32x2 odd = {(a0 >> 16) | (a1 & 0xffff0000u), (a2 >> 16) | (a3 & 0xffff0000u)};
                    const int c = cc * 8 + 2 * w;
                    *reinterpret_cast<u32x2*>(vl + c * L::V_STRIDE + 4 * kq) = even;
                    *reinterpret_cast<u32x2*>(vl + (c + 1) * L::V_STRIDE + 4 * kq) = odd;
                }
            }
        }
    };

    // ---- online-softmax state (one query row per lane) --------------------
    float m_i = -INFINITY;  // running max of scaled scores, log2 domain
    float l_i = 0.f;        // running sum of bf16-rounded probabilities (this half's keys)
    f32x16 oacc[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[cb][r] = 0.f;

    auto compute_tile = [&](const uint16_t* slot, int t) {
        const int key0 = t * BN;
        // whole tile above this wave's diagonal: nothing to do
        if (CAUSAL && key0 > q_wave0 + 31 + diag) return;
        const uint16_t* kl = slot;
        const uint16_t* vl = slot + L::K_ELEMS;

        // S^T = K Q^T
        f32x16 s[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
            const uint16_t* ka = kl + (kb * 32 + l32) * L::K_STRIDE + hh * 8;
#pragma unroll
            for (int ks = 0; ks < KD; ++ks) {
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(ka + ks * 16);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[kb], 0, 0, 0);
            }
        }

        // mask: ragged tail of the key range and, on diagonal tiles, causality
        const bool need_mask = (key0 + BN > Skv) || (CAUSAL && key0 + BN - 1 > q_wave0 + diag);
        const int lim = CAUSAL ? min(Skv - 1, qrow + diag) : Skv - 1;
        if (need_mask) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = key0 + kb * 32 + 16 * hh + r;
                    if (key > lim) s[kb][r] = -INFINITY;
                }
        }

        // row max over this tile (in-lane, then across the two wave halves)
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        // (a fully masked row gives -inf, also when the scale is 0)
        const float tmax = (mx == -INFINITY) ? -INFINITY : mx * scale_log2;
        const float m_new = fmaxf(m_i, tmax);
        const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_i - m_use);

        // probabilities, rounded to bf16 (RNE), and their sum
        bf16x8 pb[KB][2];
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    float p = __builtin_amdgcn_exp2f(fmaf(s[kb][8 * h2 + e], scale_log2, -m_use));
                    // masked keys weigh exactly 0 (their score is -inf, and -inf * 0 = NaN)
                    if (need_mask && key0 + kb * 32 + 16 * hh + 8 * h2 + e > lim) p = 0.f;
                    pb[kb][h2][e] = (__bf16)p;
                }
                const u32x4 w = __builtin_bit_cast(u32x4, pb[kb][h2]);
#pragma unroll
                for (int e = 0; e < 4; ++e) rs += bf16_lo(w[e]) + bf16_hi(w[e]);
            }
        l_i = l_i * alpha + rs;

        // rescale the output only when some row's max moved
        if (__any(m_new > m_i)) {
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
        }
        m_i = m_new;

        // O^T += V^T P^T
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            const uint16_t* va = vl + (cb * 32 + l32) * L::V_STRIDE + 16 * hh;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int h2 = 0; h2 < 2; ++h2) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(va + kb * 32 + 8 * h2);
                    oacc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kb][h2], oacc[cb], 0, 0, 0);
                }
        }
    };

    // ---- main loop over K/V tiles ------------------------------------------
    uint16_t* slot0 = lds;
    uint16_t* slot1 = lds + (DBUF ? L::SLOT : 0);
    load_tile(0);
    store_tile(slot0);
    __syncthreads();
    for (int t = 0; t < n_tiles; ++t) {
        uint16_t* cur = (DBUF && (t & 1)) ? slot1 : slot0;
        if (DBUF && t + 1 < n_tiles) load_tile(t + 1);
        compute_tile(cur, t);
        if (t + 1 < n_tiles) {
            if (DBUF) {
                store_tile((t & 1) ? slot0 : slot1);
                __syncthreads();
            } else {
                __syncthreads();
                load_tile(t + 1);
                store_tile(slot0);
                __syncthreads();
            }
        }
    }

    // ---- epilogue: O = O^T / l, one query row per lane ----------------------
    const float l_tot = l_i + __shfl_xor(l_i, 32);
    const float inv = 1.f / l_tot;
    if (qrow < Sq) {
        float* orow = O + ((long long)bh * Sq + qrow) * D + 4 * hh;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float4 val = {oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv,
                              oacc[cb][4 * g + 2] * inv, oacc[cb][4 * g + 3] * inv};
                *reinterpret_cast<float4*>(orow + cb * 32 + 8 * g) = val;
            }
    }
}

}  // namespace attn
