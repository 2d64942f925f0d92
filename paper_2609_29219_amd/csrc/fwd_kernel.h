// Prefill attention kernel for gfx950 (CDNA4).
//
// One workgroup computes BLOCK_M = 32*NW query rows of one (batch, head)
// against all allowed keys, streaming K/V in tiles of BN keys through LDS
// with an online softmax (running max m, running sum l, rescaled output).
//
// Operand orientation.  Each wave owns 32 query rows and computes the
// transposed score block S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// (A = 32 keys x 16 dims read from LDS, B = 16 dims x 32 queries held in
// VGPRs).  The 32x32 accumulator puts one query column in each lane
// (lane & 31) and 16 keys of it in that lane's 16 registers (the other 16
// keys sit in lane ^ 32).  Row max and row sum are in-lane reductions plus
// one exchange between the wave halves (v_permlane32_swap).
//
// Key permutation.  Accumulator register r of lane half h holds MFMA row
// 8*(r/4) + 4*h + r%4.  K rows are written to LDS permuted inside each
// 32-key block (LDS row p holds key 16*((p%8)/4) + 4*(p/8) + p%4), so
// register r of half h is key 16*h + r: a lane's 16 probabilities are 16
// consecutive keys, which is the k-operand layout the PV MFMA needs.
//
// PV.  O^T += V^T P^T with B = the bf16 probabilities straight from
// registers and A = V^T (32 dims x 8 keys per MFMA).  V stays row-major in
// LDS and the A operand is fetched with ds_read_b64_tr_b16: inside each
// 16-lane group, lane i addresses 4 consecutive values E[i][0..3] and lane
// 4a+b receives E[a][b], E[a+4][b], E[a+8][b], E[a+12][b].  Lane i points at
// row k0 + i/4, column base + 4*(i%4), so lane j receives the 4 keys
// k0..k0+3 of column base + j; two such reads give the 8 keys of one MFMA.
// The output accumulator holds one query per lane, so the online-softmax
// rescale is one per-lane scalar.
//
// LDS layout (64 banks of 4 bytes).  K rows are padded to D+8 bf16, so
// consecutive rows start 4 banks apart and the 16 lanes a ds_read_b128
// serves per cycle cover all 64 banks; V rows are padded to D+32 bf16, so the
// four rows a transposed read touches start 16 banks apart and its 32 lanes
// per cycle (two 16-lane groups 8 banks apart) cover all 64 banks.
//
// Pipelining (the HEG pipe knob, PIPE):
//   0  one LDS slot per operand: load -> barrier -> compute -> barrier; any
//      overlap comes from the other workgroups resident on the CU.
//   1  two slots: the global loads of tile t+1 are in flight while tile t is
//      computed, then written to the other slot; one barrier per tile.
//   2  ping-pong (8 waves): a wave cannot issue vector instructions while its
//      own MFMAs execute, but the two waves sharing a SIMD can.  Waves 0-3
//      (group A) and 4-7 (group B, one of each per SIMD) therefore run in
//      opposite phases: while A issues the MFMAs of PV(t-1) and S(t), B runs
//      the softmax of tile t on the VALU, and the other way round in the
//      second half of the tile; two barriers per tile.
// Only the tiles that hold the ragged end of the key range or cross the
// workgroup's causal diagonal run the masking code.
//
// The scale factor is strictly positive (the host maps a zero scale to the
// smallest normal float, which gives exactly equal weights), so masked scores
// of -inf always give a probability of exactly 0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// Slack (log2 units) before the running max of a row is moved.
static constexpr float kRescaleSlack = 8.0f;

template <int D, int BN>
struct FwdLds {
    static constexpr int K_STRIDE = D + 8;   // bf16 per K row
    static constexpr int V_STRIDE = D + 32;  // bf16 per V row
    static constexpr int K_TILE = BN * K_STRIDE;
    static constexpr int V_TILE = BN * V_STRIDE;
};

// LDS row of key j (0..31) inside a 32-key block; inverse of the permutation
// described above.
__device__ __forceinline__ int k_lds_row(int j) {
    return ((j >> 2) & 3) << 3 | (j >> 4) << 2 | (j & 3);
}

__device__ __forceinline__ float half_swap_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float half_swap_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ s16x4 lds_read_tr(const uint16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(p));
}

constexpr int fwd_slots(int pipe) { return pipe == 0 ? 1 : 2; }

// Waves per SIMD the register allocator should leave room for: two when two
// workgroups' LDS fits in one CU (or one 8-wave workgroup), else one.
template <int D, int BN, int NW, int PIPE>
constexpr int fwd_waves_per_eu() {
    constexpr int lds = fwd_slots(PIPE) * (FwdLds<D, BN>::K_TILE + FwdLds<D, BN>::V_TILE) * 2;
    constexpr int wgs = 163840 / lds;
    return (wgs * NW / 4) >= 2 ? 2 : 1;
}

template <int D, int BN, int NW, int PIPE, bool CAUSAL>
__global__ __launch_bounds__(NW * 64, (fwd_waves_per_eu<D, BN, NW, PIPE>())) void fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, float* __restrict__ O, int Sq, int Skv, int n_qtiles,
    int n_wg, int num_xcds, float scale_log2, uint32_t q_sign) {
    static_assert(PIPE != 2 || NW == 8, "the ping-pong schedule pairs 4 waves with 4 waves");
    constexpr int BM = NW * 32;
    constexpr int NT = NW * 64;
    constexpr int KD = D / 16;   // MFMA k-steps over the head dimension
    constexpr int KB = BN / 32;  // 32-key blocks per tile
    constexpr int CB = D / 32;   // 32-dim blocks of the output
    using L = FwdLds<D, BN>;
    constexpr int CHUNKS = BN * D / 8;  // 16-byte chunks of one K (or V) tile
    constexpr int CH = (CHUNKS + NT - 1) / NT;
    constexpr int NSLOT = fwd_slots(PIPE);

    __shared__ __attribute__((aligned(16))) uint16_t lds[NSLOT * (L::K_TILE + L::V_TILE)];
    uint16_t* const kslot0 = lds;
    uint16_t* const kslot1 = lds + (NSLOT - 1) * L::K_TILE;
    uint16_t* const vslot0 = lds + NSLOT * L::K_TILE;
    uint16_t* const vslot1 = vslot0 + (NSLOT - 1) * L::V_TILE;

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
    // Causal work grows linearly with the q-tile index, so a causal
    // workgroup takes the pair of q-tiles (n-1-u, u): every workgroup then
    // holds n+1 tiles of work (heavy one first).  Non-causal: one q-tile.
    const int units = CAUSAL ? (n_qtiles + 1) / 2 : n_qtiles;
    const int bh = logical / units;
    const int unit = logical % units;
    const int n_pass = (CAUSAL && n_qtiles - 1 - unit != unit) ? 2 : 1;
    const int diag = Skv - Sq;  // causal: key j allowed iff j <= row + diag
    const long long kv_base = (long long)bh * Skv * D;
    const uint16_t* Kb = K + kv_base;
    const uint16_t* Vb = V + kv_base;

    for (int pass = 0; pass < n_pass; ++pass) {
    const int qt = CAUSAL ? (pass == 0 ? n_qtiles - 1 - unit : unit) : unit;
    const int q_wave0 = qt * BM + wave * 32;  // first query row of this wave
    const int qrow = q_wave0 + l32;

    // ---- Q tile into VGPRs, as the B operand (16 dims x 32 queries) --------
    bf16x8 qf[KD];
    {
        // rows past Sq read the last row (finite data; never stored)
        const uint16_t* qp = Q + ((long long)bh * Sq + min(qrow, Sq - 1)) * D + hh * 8;
#pragma unroll
        for (int ks = 0; ks < KD; ++ks) {
            u32x4 w = *reinterpret_cast<const u32x4*>(qp + ks * 16);
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
    // causal: a tile entirely above this wave's diagonal is skipped
    auto wave_active = [&](int t) { return !CAUSAL || t * BN <= q_wave0 + 31 + diag; };
    // tiles before first_masked need no mask for any row of this workgroup
    int first_masked = Skv / BN;  // the ragged tail tile, if any
    if (CAUSAL) first_masked = min(first_masked, (qt * BM + diag + 1) / BN);

    // Rows past the end of the key range are loaded from the last valid row
    // (clamped, never out of bounds): their scores are masked to weight 0,
    // and their V values are finite, so they contribute exactly 0.
    auto load_rows = [&](const uint16_t* base, int t, u32x4 (&reg)[CH]) {
        const int key0 = t * BN;
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int u = tid + i * NT;
            if (CHUNKS % NT == 0 || u < CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                const int key = min(key0 + j, Skv - 1);
                reg[i] = *reinterpret_cast<const u32x4*>(base + (long long)key * D + cc * 8);
            }
        }
    };
    auto store_k = [&](uint16_t* dst, const u32x4 (&reg)[CH]) {
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int u = tid + i * NT;
            if (CHUNKS % NT == 0 || u < CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                const int prow = (j & ~31) | k_lds_row(j & 31);
                *reinterpret_cast<u32x4*>(dst + prow * L::K_STRIDE + cc * 8) = reg[i];
            }
        }
    };
    auto store_v = [&](uint16_t* dst, const u32x4 (&reg)[CH]) {
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int u = tid + i * NT;
            if (CHUNKS % NT == 0 || u < CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                *reinterpret_cast<u32x4*>(dst + j * L::V_STRIDE + cc * 8) = reg[i];
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

    // S^T = K Q^T for one tile (independent accumulators interleaved).
    auto scores = [&](const uint16_t* kl, f32x16 (&s)[KB]) {
        const uint16_t* ka_base = kl + l32 * L::K_STRIDE + hh * 8;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KD; ++ks)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                const bf16x8 a = *reinterpret_cast<const bf16x8*>(ka_base + kb * 32 * L::K_STRIDE + ks * 16);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[kb], 0, 0, 0);
            }
    };

    // Online-softmax statistics of tile t: mask (MASK tiles only), row max,
    // and the lazy rescale.  The running max m_i of a row only moves when the
    // tile's max exceeds it by more than kRescaleSlack (log2 units), so the
    // output rescale is skipped on almost every tile; probabilities are then
    // bounded by 2^kRescaleSlack, and the numerator and the normaliser share
    // the same reference, so the result is unchanged.  Returns the reference
    // to subtract.
    auto softmax_stats = [&](f32x16 (&s)[KB], int t, auto mask_tag) -> float {
        constexpr bool MASK = decltype(mask_tag)::value;
        const int key0 = t * BN;
        if (MASK) {
            // ragged tail of the key range and, on diagonal tiles, causality:
            // register r of block kb holds key key0 + 16*hh + (kb*32 + r), so
            // compare the constant kb*32 + r against one per-lane bound
            const int lim = CAUSAL ? min(Skv - 1, qrow + diag) : Skv - 1;
            const int room = lim - key0 - 16 * hh;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (kb * 32 + r > room) s[kb][r] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
        mx = half_swap_max(mx);
        const float tmax = (mx == -INFINITY) ? -INFINITY : mx * scale_log2;
        const bool move = tmax > m_i + kRescaleSlack;  // also true for the first finite max
        if (__any(move)) {
            const float m_new = move ? tmax : m_i;
            const float alpha = __builtin_amdgcn_exp2f(m_i - m_new);  // 0 when m_i = -inf
            l_i *= alpha;
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
            m_i = m_new;
        }
        return (m_i == -INFINITY) ? 0.f : m_i;
    };
    // bf16 probabilities of a tile and their sum (VALU only).  Masked scores
    // are -inf and the scale is > 0, so they give exactly 0.
    auto probs = [&](const f32x16 (&s)[KB], float m_ref, bf16x8 (&pb)[KB][2]) {
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    pb[kb][h2][e] =
                        (__bf16)__builtin_amdgcn_exp2f(fmaf(s[kb][8 * h2 + e], scale_log2, -m_ref));
                // sum of the rounded probabilities (bf16 -> fp32 is a shift or a
                // mask); plain adds co-issue with another wave's MFMAs, which the
                // bf16 dot-product instructions do not
                const u32x4 w = __builtin_bit_cast(u32x4, pb[kb][h2]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    rs += __uint_as_float(w[e] << 16) + __uint_as_float(w[e] & 0xffff0000u);
            }
        l_i += rs;
    };

    // O^T += V^T P^T in groups of 8 keys; V^T operands by transposed reads.
    const int tr_row = (lane & 15) >> 2;                         // + k0
    const int tr_col = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);  // + cb*32
    auto pv = [&](const uint16_t* vl, const bf16x8 (&pb)[KB][2]) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const uint16_t* p =
                    vl + (kb * 32 + 16 * hh + 8 * h2 + tr_row) * L::V_STRIDE + tr_col;
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) {
                    const s16x4 lo = lds_read_tr(p + cb * 32);
                    const s16x4 hi = lds_read_tr(p + cb * 32 + 4 * L::V_STRIDE);
                    const s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                    oacc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8, w), pb[kb][h2], oacc[cb], 0, 0, 0);
                }
            }
    };

    // ---- main loop over K/V tiles ------------------------------------------
    // Every schedule runs its tiles in two loops: first the tiles that need no
    // mask, then the masked ones (compile-time tag), so the masking code never
    // sits in the common loop body.
    auto two_loops = [&](int t0, auto&& step) {
        int t = t0;
        const int split = max(t0, min(first_masked, n_tiles));
        for (; t < split; ++t) step(t, std::false_type{});
        for (; t < n_tiles; ++t) step(t, std::true_type{});
    };
    u32x4 kr[CH], vr[CH];
    if (PIPE == 0) {
        two_loops(0, [&](int t, auto mask_tag) {
            load_rows(Kb, t, kr);
            load_rows(Vb, t, vr);
            store_k(kslot0, kr);
            store_v(vslot0, vr);
            __syncthreads();
            if (wave_active(t)) {
                f32x16 s[KB];
                bf16x8 pb[KB][2];
                scores(kslot0, s);
                probs(s, softmax_stats(s, t, mask_tag), pb);
                pv(vslot0, pb);
            }
            __syncthreads();
        });
    } else if (PIPE == 1) {
        // tile t+1 is fetched into registers while tile t is computed from
        // LDS, then written to the other slot; one barrier per tile
        load_rows(Kb, 0, kr);
        load_rows(Vb, 0, vr);
        store_k(kslot0, kr);
        store_v(vslot0, vr);
        __syncthreads();
        two_loops(0, [&](int t, auto mask_tag) {
            const bool odd = t & 1;
            if (t + 1 < n_tiles) {
                load_rows(Kb, t + 1, kr);
                load_rows(Vb, t + 1, vr);
            }
            if (wave_active(t)) {
                f32x16 s[KB];
                bf16x8 pb[KB][2];
                scores(odd ? kslot1 : kslot0, s);
                probs(s, softmax_stats(s, t, mask_tag), pb);
                pv(odd ? vslot1 : vslot0, pb);
            }
            if (t + 1 < n_tiles) {
                store_k(odd ? kslot0 : kslot1, kr);
                store_v(odd ? vslot0 : vslot1, vr);
            }
            __syncthreads();
        });
    } else {
        // Ping-pong.  LDS holds K_t, K_{t+1} and V_{t-1}, V_t in two-slot
        // rings (tile t in slot t&1).  Per tile t:
        //   phase 1: A: PV(t-1), S(t)          B: softmax(t)
        //   phase 2: A: softmax(t)             B: PV(t), S(t+1)
        // The global loads of K_{t+2} and V_{t+1} are issued at the start of
        // phase 1 and written to LDS at the end of phase 2 (into the slots of
        // K_t and V_{t-1}, whose last readers finished in phase 1).
        const bool group_b = wave >= 4;
        f32x16 s[KB];
        bf16x8 pb[KB][2];
        bool pv_pending = false;  // group A: PV of the previous tile is due
        load_rows(Kb, 0, kr);
        load_rows(Vb, 0, vr);
        store_k(kslot0, kr);
        store_v(vslot0, vr);
        if (n_tiles > 1) {
            load_rows(Kb, 1, kr);
            store_k(kslot1, kr);
        }
        __syncthreads();
        if (group_b && wave_active(0)) scores(kslot0, s);
        two_loops(0, [&](int t, auto mask_tag) {
            const bool odd = t & 1;
            uint16_t* const k_t = odd ? kslot1 : kslot0;
            uint16_t* const k_t1 = odd ? kslot0 : kslot1;
            uint16_t* const v_t = odd ? vslot1 : vslot0;
            uint16_t* const v_t1 = odd ? vslot0 : vslot1;  // holds V_{t-1}
            if (t + 2 < n_tiles) load_rows(Kb, t + 2, kr);
            if (t + 1 < n_tiles) load_rows(Vb, t + 1, vr);
            // phase 1
            if (!group_b) {
                if (pv_pending) pv(v_t1, pb);
                pv_pending = false;
                if (wave_active(t)) scores(k_t, s);
            } else if (wave_active(t)) {
                probs(s, softmax_stats(s, t, mask_tag), pb);
            }
            __syncthreads();
            // phase 2
            if (!group_b) {
                if (wave_active(t)) {
                    probs(s, softmax_stats(s, t, mask_tag), pb);
                    pv_pending = true;
                }
            } else if (wave_active(t)) {
                pv(v_t, pb);
                if (t + 1 < n_tiles && wave_active(t + 1)) scores(k_t1, s);
            }
            if (t + 2 < n_tiles) store_k(k_t, kr);
            if (t + 1 < n_tiles) store_v(v_t1, vr);
            __syncthreads();
        });
        if (pv_pending) pv(((n_tiles - 1) & 1) ? vslot1 : vslot0, pb);
    }

    // ---- epilogue: O = O^T / l, one query row per lane ----------------------
    const float inv = 1.f / half_swap_sum(l_i);
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
    __syncthreads();  // the next q-tile refills LDS slots read above
    }  // pass
}

}  // namespace attn
