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
// keys sit in lane ^ 32).  The row max is an in-lane reduction plus one
// exchange between the wave halves (v_permlane32_swap); the row sum is taken
// by the matrix core (below).
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
// Row sums.  The normaliser (the running sum of the bf16 probabilities) is
// accumulated on the matrix core too, with one v_mfma_f32_16x16x32_bf16 per
// 16-key step: its B operand is the PV MFMA's probability register read as a
// 32 x 16 matrix (lane l holds k-group l/16, column l%16), so k-groups 0 and 2
// are the 16 keys of query c = l%16 and k-groups 1 and 3 those of query c+16.
// A is a constant 0/1 selector with A[i][k] = 1 iff (k/8)%2 == (i/4)%2, so the
// output rows 4g..4g+3 that lane l holds (g = l/16) sum the keys of query
// c + 16*(g%2) = l%32: each lane gets the row sum of its own query, in the
// same lane as its output accumulator, with no exchange between lanes.  This
// replaces four VALU instructions per pair of probabilities; the variants
// already at the 256-register limit keep the VALU sum (fwd_mfma_row_sum).
//
// LDS layout (64 banks of 4 bytes).  K rows are padded to D+8 bf16, so
// consecutive rows start 4 banks apart and the 16 lanes a ds_read_b128
// serves per cycle cover all 64 banks; V rows are padded to D+32 bf16, so the
// four rows a transposed read touches start 16 banks apart and its 32 lanes
// per cycle (two 16-lane groups 8 banks apart) cover all 64 banks.
//
// Tile loads.  Pipes 0, 1 and 3 load K/V tiles straight from global memory
// into LDS (buffer_load_dwordx4 ... lds), with the K permutation and the
// padding expressed in the per-lane source addresses; pipe 2 stages them
// through registers.  With two slots (pipes 1 and 3) the LDS loads are
// issued from inline assembly (lds_dma.h) and every workgroup barrier first
// waits for the wave's own loads: issued through the compiler builtin, they
// made the compiler hold reads of the current tile until the next tile's
// loads had landed.  Pipe 0 has one slot, nothing to overlap, and keeps the
// builtin.
//
// Pipelining (the HEG pipe knob, PIPE):
//   0  one LDS slot per operand: load -> barrier -> compute -> barrier; any
//      overlap comes from the other workgroups resident on the CU.
//   1  two slots: tile t+1 streams into the other slot while tile t is
//      computed; one barrier per tile.
//   2  ping-pong (8 waves): waves 0-3 (group A) and 4-7 (group B, one of each
//      per SIMD) run in opposite phases: while A issues the MFMAs of PV(t-1)
//      and S(t), B runs the softmax of tile t on the VALU, and the other way
//      round in the second half of the tile; two barriers per tile.
//   3  software pipeline: each wave issues the MFMAs of S(t+1) and PV(t) one
//      by one with the softmax VALU work of tile t between them (a wave issues
//      in order, so the matrix core and the VALU work together only if the
//      instruction stream interleaves them); one barrier per tile.
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

#include "common.h"
#include "lds_dma.h"

namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// Slack (log2 units) before the running max of a row is moved.
static constexpr float kRescaleSlack = 8.0f;
static constexpr float kLn2 = 0.69314718055994531f;

template <int D, int BN>
struct FwdLds {
    static constexpr int K_STRIDE = D + 8;   // bf16 per K row
    static constexpr int V_STRIDE = D + 32;  // bf16 per V row
    // slot sizes rounded up to whole 1 KiB pieces of the direct tile loads
    static constexpr int K_TILE = fwd_k_slot_elems(D, BN);
    static constexpr int V_TILE = fwd_v_slot_elems(D, BN);
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

// Row sums on the matrix core (8 more registers per wave: the selector and
// the accumulator) everywhere but in the d = 128 kernels that would then
// spill: 128-key tiles, and the four-wave software pipeline.
constexpr bool fwd_mfma_row_sum(int d, int bn, int nw, int pipe) {
    return !(d == 128 && (bn == 128 || (nw == 4 && pipe == 3)));
}

// Entries of the software pipeline's LDS operand ring (operands are fetched
// PF - 1 MFMAs ahead): two in the causal kernels, which need the registers
// for their masks and the row-sum MFMA (and measured as fast with two),
// three elsewhere (more measured no faster).
constexpr int fwd_operand_ring(bool causal) { return causal ? 2 : 3; }

// Software-pipeline lag (0 to max_lag slots) between the exponentials of a
// probability pair and its rounding: the largest for which every pair is
// still rounded in a slot before the first PV MFMA of its 16-key step (the
// pair's work follows the slot's MFMA in program order); -1 if even lag 0
// violates that.
constexpr int fwd_pair_lag(int npair, int exp_slots, int ns, int cb, int max_lag = 2) {
    for (int lag = max_lag; lag >= 0; --lag) {
        bool ok = true;
        for (int pp = 0; pp < npair; ++pp)
            if (pp * exp_slots / npair + lag >= ns + (pp / 4) * cb) ok = false;
        if (ok) return lag;
    }
    return -1;
}

// Waves per SIMD the register allocator should leave room for: two when two
// workgroups' LDS fits in one CU (or one 8-wave workgroup), else one.
template <int D, int BN, int NW, int PIPE>
constexpr int fwd_waves_per_eu() {
    constexpr int lds = fwd_lds_bytes(D, BN, PIPE, NW);
    constexpr int wgs = 163840 / lds;
    return (wgs * NW / 4) >= 2 ? 2 : 1;
}

template <int D, int BN, int NW, int PIPE, bool CAUSAL>
__global__ __launch_bounds__(NW * 64, (fwd_waves_per_eu<D, BN, NW, PIPE>())) void fwd_kernel(
    const FwdArgs args) {
    const uint16_t* __restrict__ Q = args.q;
    const uint16_t* __restrict__ K = args.k;
    const uint16_t* __restrict__ V = args.v;
    const int Sq = args.Sq, n_qtiles = args.n_qtiles, n_wg = args.n_wg;
    const int num_xcds = args.num_xcds;
    const float scale_log2 = args.scale_log2;
    const uint32_t q_sign = args.q_sign;
    static_assert(PIPE != 2 || NW == 8, "the ping-pong schedule pairs 4 waves with 4 waves");
    static_assert(PIPE != 3 || BN <= 64, "two score tiles in registers");
    constexpr int BM = NW * 32;
    constexpr int NT = NW * 64;
    constexpr int KD = D / 16;   // MFMA k-steps over the head dimension
    constexpr int KB = BN / 32;  // 32-key blocks per tile
    constexpr int CB = D / 32;   // 32-dim blocks of the output
    using L = FwdLds<D, BN>;
    constexpr int CHUNKS = BN * D / 8;  // 16-byte chunks of one K (or V) tile
    constexpr int CH = (CHUNKS + NT - 1) / NT;
    constexpr int NSLOT = fwd_slots(PIPE);

    static_assert(fwd_lds_bytes(D, BN, PIPE, NW) >= NSLOT * (L::K_TILE + L::V_TILE) * 2, "");
    __shared__ __attribute__((aligned(16))) uint16_t lds[fwd_lds_bytes(D, BN, PIPE, NW) / 2];
    uint16_t* const kslot0 = lds;
    uint16_t* const kslot1 = lds + (NSLOT - 1) * L::K_TILE;
    uint16_t* const vslot0 = lds + NSLOT * L::K_TILE;
    uint16_t* const vslot1 = vslot0 + (NSLOT - 1) * L::V_TILE;

    // Workgroup barrier.  Pipes 1 and 3 issue their LDS loads from inline
    // assembly, which the compiler does not track: each wave first waits for
    // its own loads, so the barrier publishes them.  Pipe 0 (one slot) and
    // pipe 2 (stores from registers) keep the compiler's barrier.
    auto tile_barrier = [&]() __attribute__((always_inline)) {
        if constexpr (PIPE == 1 || PIPE == 3)
            publish_barrier<0>();
        else
            __syncthreads();
    };

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar
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
    // holds n+1 tiles of work (heavy one first).  Non-causal: one q-tile,
    // of one key split (logical = (head, split, q-tile), q-tile fastest, so
    // the workgroups reading one K/V chunk are neighbours on one XCD).
    const int units = CAUSAL ? (n_qtiles + 1) / 2 : n_qtiles;
    const int kv_splits = (CAUSAL || PIPE == 2) ? 1 : args.kv_splits;
    const int bh = logical / (units * kv_splits);
    const int within = logical - bh * units * kv_splits;
    const int split = within / units;
    const int unit = within - split * units;
    const int n_pass = (CAUSAL && n_qtiles - 1 - unit != unit) ? 2 : 1;
    // this workgroup's keys: [k0, k0 + Skv) of the head's args.Skv keys
    const int k0 = split * args.kv_chunk;
    const int Skv = CAUSAL ? args.Skv : min(args.kv_chunk, args.Skv - k0);
    const int diag = Skv - Sq;  // causal: key j allowed iff j <= row + diag
    // grouped-query heads: query head bh reads key/value head bh / group
    const long long kv_base = ((long long)(bh / args.group) * args.Skv + k0) * D;
    const uint16_t* Kb = K + kv_base;
    const uint16_t* Vb = V + kv_base;

    auto qt_of = [&](int pass) __attribute__((always_inline)) {
        return CAUSAL ? (pass == 0 ? n_qtiles - 1 - unit : unit) : unit;
    };
    // ---- Q tile into VGPRs, as the B operand (16 dims x 32 queries) ----------
    // The loads are issued without touching the data, so nothing waits for
    // them until the first MFMA that reads Q (the tile loads of the first K/V
    // tiles, or the previous q-tile's epilogue, go on meanwhile).  A negative
    // scale is applied by flipping the sign bits of Q (exact) at the start of
    // the pass, only when it is negative.
    bf16x8 qf[KD];
    auto load_q = [&](int qt) __attribute__((always_inline)) {
        // rows past Sq read the last row (finite data; never stored)
        const int row = min(qt * BM + wave * 32 + l32, Sq - 1);
        const uint16_t* qp = Q + ((long long)bh * Sq + row) * D + hh * 8;
#pragma unroll
        for (int ks = 0; ks < KD; ++ks)
            qf[ks] = *reinterpret_cast<const bf16x8*>(qp + ks * 16);
    };
    load_q(qt_of(0));

    for (int pass = 0; pass < n_pass; ++pass) {
    if (q_sign) {
#pragma unroll
        for (int ks = 0; ks < KD; ++ks)
            qf[ks] = __builtin_bit_cast(bf16x8, __builtin_bit_cast(u32x4, qf[ks]) ^ q_sign);
    }
    const int qt = qt_of(pass);
    const int q_wave0 = qt * BM + wave * 32;  // first query row of this wave
    const int qrow = q_wave0 + l32;

    // ---- key range of this workgroup ------------------------------------
    int kv_end = Skv;
    if (CAUSAL) {
        const int last_q = min(qt * BM + BM - 1, Sq - 1);
        kv_end = min(Skv, last_q + diag + 1);
    }
    const int n_tiles = (kv_end + BN - 1) / BN;
    // causal: a tile entirely above this wave's diagonal is skipped
    auto wave_active = [&](int t) __attribute__((always_inline)) { return !CAUSAL || t * BN <= q_wave0 + 31 + diag; };
    // tiles before first_masked need no mask for any row of this wave.  The
    // split is per wave (on the diagonal, the waves of lower rows start
    // masking earlier); every wave still runs one barrier per tile.
    int first_masked = Skv / BN;  // the ragged tail tile, if any
    if (CAUSAL) first_masked = min(first_masked, (q_wave0 + diag + 1) / BN);

    // Rows past the end of the key range are loaded from the last valid row
    // (clamped, never out of bounds): their scores are masked to weight 0,
    // and their V values are finite, so they contribute exactly 0.
    auto load_rows = [&](const uint16_t* base, int t, u32x4 (&reg)[CH]) __attribute__((always_inline)) {
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
    auto store_k = [&](uint16_t* dst, const u32x4 (&reg)[CH]) __attribute__((always_inline)) {
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
    auto store_v = [&](uint16_t* dst, const u32x4 (&reg)[CH]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int u = tid + i * NT;
            if (CHUNKS % NT == 0 || u < CHUNKS) {
                const int j = u / (D / 8), cc = u % (D / 8);
                *reinterpret_cast<u32x4*>(dst + j * L::V_STRIDE + cc * 8) = reg[i];
            }
        }
    };

    // Direct global -> LDS tile loads (pipes 0, 1, 3) with buffer_load ... lds:
    // lane i of an instruction writes its 16 bytes at the wave-uniform LDS base
    // + 16*i, so a tile region (its padded rows laid end to end) is filled in
    // 1 KiB pieces, and each lane picks the source chunk that belongs at its
    // position: the K row permutation and the padding live in the source
    // offsets (a padding position re-reads a chunk of its own row).  The
    // buffer resource holds this head's K or V slab (reads past it return 0),
    // the tile base is a scalar offset and each lane's offset within the tile
    // is fixed, so issuing a tile costs no vector arithmetic and no registers
    // carry tile data; the loads complete behind the barrier that publishes
    // them.
    constexpr int DCH = D / 8;                                   // 16-byte chunks of a row
    constexpr int KST = L::K_STRIDE / 8, VST = L::V_STRIDE / 8;  // per padded LDS row
    constexpr int KCH = BN * KST, VCH = BN * VST;                // positions per region
    constexpr int KI = (KCH + 63) / 64, VI = (VCH + 63) / 64;    // pieces per region
    constexpr int NJK = (KI + NW - 1) / NW, NJV = (VI + NW - 1) / NW;  // pieces per wave
    const uint32_t slab_bytes = (uint32_t)Skv * D * 2;  // fits in 31 bits (checked by the host)
    const dma_rsrc_t k_rsrc = make_dma_rsrc(Kb, slab_bytes);
    const dma_rsrc_t v_rsrc = make_dma_rsrc(Vb, slab_bytes);
    constexpr int kRsrcFlags = 0x00020000;  // raw 32-bit buffer, gfx9 family
    const __amdgpu_buffer_rsrc_t k_rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Kb), 0, (int)slab_bytes, kRsrcFlags);
    const __amdgpu_buffer_rsrc_t v_rsrc_b = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Vb), 0, (int)slab_bytes, kRsrcFlags);
    // LDS byte address of the slots: the array's, plus element offsets
    const uint32_t lds_base = lds_address(lds);
    // K piece p (0 <= p < KI) goes to wave p % NW, and so does V piece p
    // (0 <= p < VI): the K/V choice of a piece is known at compile time and
    // whether it exists is a scalar test on the wave index (only for a
    // wave's last piece of each operand).  offk[j], offv[j]: byte offset
    // inside a tile of this lane's source chunk for the wave's j-th K or V
    // piece.  Where a region ends inside its last piece, the lanes past its
    // end fill the slot's padding (slots are whole pieces) with a copy of the
    // region's last chunk, so no lane is masked off.
    static_assert(L::K_TILE * 2 >= KI * 1024 && L::V_TILE * 2 >= VI * 1024, "");
    auto src_offset = [&](auto is_k_tag, int i) __attribute__((always_inline)) -> int {
        constexpr bool IS_K = decltype(is_k_tag)::value;
        const int pos = min(i * 64 + lane, (IS_K ? KCH : VCH) - 1);
        constexpr int st = IS_K ? KST : VST;
        const int prow = pos / st, c = min(pos % st, DCH - 1);
        const int key = IS_K ? (prow & ~31) | (16 * ((prow & 7) >> 2) + 4 * ((prow & 31) >> 3) +
                                              (prow & 3))
                             : prow;
        return (key * D + c * 8) * 2;
    };
    int offk[NJK], offv[NJV];
#pragma unroll
    for (int j = 0; j < NJK; ++j) offk[j] = src_offset(std::true_type{}, wave + j * NW);
#pragma unroll
    for (int j = 0; j < NJV; ++j) offv[j] = src_offset(std::false_type{}, wave + j * NW);
    // The wave's pieces of one operand of tile t into the slot at element
    // offset dst0 of the LDS array.  Slots are named by integer offsets:
    // generic-pointer arithmetic on LDS addresses here made the backend emit
    // an invalid null check.
    auto dma_operand = [&](auto is_k_tag, int t, int dst0) __attribute__((always_inline)) {
        constexpr bool IS_K = decltype(is_k_tag)::value;
        constexpr int NI = IS_K ? KI : VI, NJO = IS_K ? NJK : NJV;
        const int key0 = t * BN;
        auto pieces = [&](auto ragged_tag) __attribute__((always_inline)) {
#pragma unroll
            for (int j = 0; j < NJO; ++j) {
                const int i = wave + j * NW;
                if ((j + 1) * NW > NI && i >= NI) continue;  // scalar; only the last piece
                int o = IS_K ? offk[j] : offv[j];
                if (ragged_tag)  // rows past the end re-read the last key
                    o = ((min(key0 + o / (2 * D), Skv - 1) - key0) * D) * 2 + o % (2 * D);
                const uint32_t dst = lds_base + (uint32_t)(dst0 + i * 512) * 2;
                if constexpr (PIPE == 0) {
                    // one slot: no read overlaps a load, the builtin's waits cost nothing
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        IS_K ? k_rsrc_b : v_rsrc_b,
                        (__attribute__((address_space(3))) void*)(uintptr_t)dst, 16, o,
                        key0 * D * 2, 0, 0);
                } else {
                    lds_dma16(IS_K ? k_rsrc : v_rsrc, dst, o, key0 * D * 2);
                }
            }
        };
        // the ragged tail tile in a branch of its own, so the common path
        // issues its loads without any offset arithmetic (the causal kernels
        // keep the compiler's select form: the second copy of the loads would
        // push the software-pipelined one past its 256 registers)
        if constexpr (CAUSAL) {
            pieces(key0 + BN > Skv);
        } else {
            if (key0 + BN > Skv)
                pieces(std::true_type{});
            else
                pieces(std::false_type{});
        }
    };
    // Issue this wave's pieces of K tile tk (into the K slot at kdst) and/or
    // V tile tv (into the V slot at vdst); a negative tile index skips that
    // operand.
    auto dma = [&](int tk, int kdst, int tv, int vdst) __attribute__((always_inline)) {
        if (tk >= 0) dma_operand(std::true_type{}, tk, kdst);
        if (tv >= 0) dma_operand(std::false_type{}, tv, vdst);
    };
    // element offsets of the slots in the LDS array
    constexpr int KS0 = 0, KS1 = (NSLOT - 1) * L::K_TILE;
    constexpr int VS0 = NSLOT * L::K_TILE, VS1 = VS0 + (NSLOT - 1) * L::V_TILE;
    auto dma_k = [&](int t, int dst) __attribute__((always_inline)) {
        dma(t, dst, -1, dst);  // the V destination is unused
    };

    // ---- online-softmax state (one query row per lane) --------------------
    float m_i = -INFINITY;  // running max of scaled scores, log2 domain
    // Running sum of the row's bf16 probabilities: on the matrix core (all
    // four registers of lsum hold it; lsum += sel * P^T per 16-key step, sel
    // the constant 0/1 selector described at the top of the file), or on the
    // VALU in l_i (this lane's half of the keys).
    constexpr bool MSUM = fwd_mfma_row_sum(D, BN, NW, PIPE);
    float l_i = 0.f;
    f32x4 lsum = {0.f, 0.f, 0.f, 0.f};
    bf16x8 sel;
    if constexpr (MSUM) {
        const __bf16 v = ((lane >> 4) & 1) == ((lane >> 2) & 1) ? (__bf16)1.0f : (__bf16)0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) sel[e] = v;
    }
    auto row_sum = [&](const bf16x8& p) __attribute__((always_inline)) {
        if constexpr (MSUM) lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, p, lsum, 0, 0, 0);
    };
    f32x16 oacc[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[cb][r] = 0.f;

    // S^T = K Q^T for one tile (independent accumulators interleaved).
    auto scores = [&](const uint16_t* kl, f32x16 (&s)[KB]) __attribute__((always_inline)) {
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

    // Row max of a tile's scores (masked in place on MASK tiles: the ragged
    // end of the key range and, on diagonal tiles, causality).  Register r of
    // block kb holds key key0 + 16*hh + (kb*32 + r), so the constant kb*32 + r
    // is compared against one per-lane bound.
    auto tile_max = [&](f32x16 (&s)[KB], int t, auto mask_tag) __attribute__((always_inline)) -> float {
        constexpr bool MASK = decltype(mask_tag)::value;
        if (MASK) {
            const int lim = CAUSAL ? min(Skv - 1, qrow + diag) : Skv - 1;
            const int room = lim - t * BN - 16 * hh;
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
        return half_swap_max(mx);
    };
    // Lazy rescale: the running max m_i of a row only moves when a tile's max
    // exceeds it by more than kRescaleSlack (log2 units), so the output
    // rescale is skipped on almost every tile; probabilities are then bounded
    // by 2^kRescaleSlack, and the numerator and the normaliser share the same
    // reference, so the result is unchanged.  Returns the reference to
    // subtract (0 while the row has seen no allowed key).
    auto update_ref = [&](float mx) __attribute__((always_inline)) -> float {
        const float tmax = (mx == -INFINITY) ? -INFINITY : mx * scale_log2;
        const bool move = tmax > m_i + kRescaleSlack;  // also true for the first finite max
        if (__any(move)) {
            const float m_new = move ? tmax : m_i;
            const float alpha = __builtin_amdgcn_exp2f(m_i - m_new);  // 0 when m_i = -inf
            if constexpr (MSUM)
                lsum *= alpha;
            else
                l_i *= alpha;
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
            m_i = m_new;
        }
        return (m_i == -INFINITY) ? 0.f : m_i;
    };
    auto softmax_stats = [&](f32x16 (&s)[KB], int t, auto mask_tag) __attribute__((always_inline)) -> float {
        return update_ref(tile_max(s, t, mask_tag));
    };
    // bf16 probabilities of a tile (VALU only).  The normaliser sums these
    // rounded values (row_sum next to the PV MFMAs that apply them, or here
    // on the VALU, where bf16 -> fp32 is a shift or a mask), so the weights
    // applied to V sum exactly to the normaliser: the output is a convex
    // combination of V rows up to fp32 rounding.  Masked scores are -inf and
    // the scale is > 0, so they give exactly 0.
    auto rounded_pair = [&](float x0, float x1, bf16x8& dst, int e, float& r0, float& r1)
        __attribute__((always_inline)) {
        // one packed conversion (the VALU sum reads both halves back from it)
        const bf16x2 pk = {(__bf16)x0, (__bf16)x1};
        dst[e] = pk[0];
        dst[e + 1] = pk[1];
        if constexpr (!MSUM) {
            const uint32_t w = __builtin_bit_cast(uint32_t, pk);
            r0 += __uint_as_float(w << 16);
            r1 += __uint_as_float(w & 0xffff0000u);
        }
    };
    auto probs = [&](const f32x16 (&s)[KB], float m_ref, bf16x8 (&pb)[KB][2])
        __attribute__((always_inline)) {
        float rs0 = 0.f, rs1 = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
                for (int e = 0; e < 8; e += 2)
                    rounded_pair(
                        __builtin_amdgcn_exp2f(fmaf(s[kb][8 * h2 + e], scale_log2, -m_ref)),
                        __builtin_amdgcn_exp2f(fmaf(s[kb][8 * h2 + e + 1], scale_log2, -m_ref)),
                        pb[kb][h2], e, rs0, rs1);
        if constexpr (!MSUM) l_i += rs0 + rs1;
    };

    // O^T += V^T P^T in steps of 16 keys (and the row sums of P); V^T
    // operands by transposed reads.
    const int tr_row = (lane & 15) >> 2;                         // + k0
    const int tr_col = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);  // + cb*32
    auto pv = [&](const uint16_t* vl, const bf16x8 (&pb)[KB][2]) __attribute__((always_inline)) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                row_sum(pb[kb][h2]);
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

    // One tile t of the software pipeline.  The MFMAs of S(t+1) (K_{t+1}
    // from kl, into s_nxt; HAS_S only) and then of PV(t) (V_t from vl) are
    // issued one by one; between them, in program order, sit the
    // exponentials of tile t (scores s_cur, reference m_ref, probabilities
    // into pb) and, once S(t+1) is complete, the row max of tile t+1 (masked
    // in place first on MASK_NEXT tiles), which is returned.  Probabilities of
    // a 16-key step are produced before the PV MFMAs that consume them.  LDS
    // operands come from a PF-entry ring, fetched PF - 1 MFMAs ahead (deeper
    // rings measured no faster), which also bounds their registers.
    auto fused_tile = [&](const uint16_t* kl, const uint16_t* vl, const f32x16 (&s_cur)[KB],
                          f32x16 (&s_nxt)[KB], bf16x8 (&pb)[KB][2], int t, float m_ref,
                          auto has_s_tag, auto mask_tag) __attribute__((always_inline)) -> float {
        constexpr bool HAS_S = decltype(has_s_tag)::value;
        constexpr bool MASK_NEXT = decltype(mask_tag)::value;
        constexpr int NS = HAS_S ? KB * KD : 0;  // MFMAs of S(t+1)
        constexpr int NPV = KB * 2 * CB;          // MFMAs of PV(t)
        constexpr int NM = NS + NPV;
        constexpr int PF = fwd_operand_ring(CAUSAL);
        constexpr int NPAIR = KB * 8;                    // pairs of probabilities per lane
        constexpr int EXP_SLOTS = HAS_S ? NS + NPV / 2 : 0;  // slots carrying exponentials
        constexpr int MAX0 = EXP_SLOTS + 1;              // first slot carrying the next max
        constexpr int NMAXV = HAS_S ? KB * 16 : 0;      // scores of tile t+1 per lane
        static_assert(!HAS_S || MAX0 < NM, "too few MFMAs to carry the softmax");
        // The exponentials of pair pp (16-key step pp / 4) are taken in slot
        // pp * EXP_SLOTS / NPAIR and rounded (and, with VALU row sums,
        // summed) LAG slots later, so the rounding does not wait on a
        // just-issued exponential; the rounded pair must still precede the
        // first PV MFMA of its step, in slot NS + (pp / 4) * CB.
        // (not with four waves: their 64-key kernel then spills).  At most one
        // slot where the rounding is a single conversion (row sums on the
        // matrix core) and the kernel is not causal; two elsewhere (measured).
        constexpr int LAG = HAS_S && NW == 8
                                ? fwd_pair_lag(NPAIR, EXP_SLOTS, NS, CB, MSUM && !CAUSAL ? 1 : 2)
                                : 0;
        static_assert(!HAS_S || fwd_pair_lag(NPAIR, EXP_SLOTS, NS, CB) >= 0,
                      "probabilities must precede their PV MFMAs");
        auto fetch = [&](int i) __attribute__((always_inline)) -> bf16x8 {
            if (i < NS) {
                const int ks = i / KB, kb = i % KB;
                return *reinterpret_cast<const bf16x8*>(kl + (kb * 32 + l32) * L::K_STRIDE +
                                                        hh * 8 + ks * 16);
            }
            const int j = i - NS, kb = j / (2 * CB), h2 = (j / CB) % 2, cb = j % CB;
            const uint16_t* p =
                vl + (kb * 32 + 16 * hh + 8 * h2 + tr_row) * L::V_STRIDE + tr_col + cb * 32;
            const s16x4 lo = lds_read_tr(p);
            const s16x4 hi = lds_read_tr(p + 4 * L::V_STRIDE);
            const s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            return __builtin_bit_cast(bf16x8, w);
        };
        float mx = -INFINITY, rs0 = 0.f, rs1 = 0.f;
        float xe[NPAIR][2];  // exponentials waiting LAG slots for rounding
        auto exps = [&](int pp) __attribute__((always_inline)) {
            const int kb = pp / 8, h2 = (pp / 4) % 2, e = 2 * (pp % 4);
            xe[pp][0] = __builtin_amdgcn_exp2f(fmaf(s_cur[kb][8 * h2 + e], scale_log2, -m_ref));
            xe[pp][1] = __builtin_amdgcn_exp2f(fmaf(s_cur[kb][8 * h2 + e + 1], scale_log2, -m_ref));
        };
        auto round_sum = [&](int pp) __attribute__((always_inline)) {
            const int kb = pp / 8, h2 = (pp / 4) % 2, e = 2 * (pp % 4);
            rounded_pair(xe[pp][0], xe[pp][1], pb[kb][h2], e, rs0, rs1);
        };
        if (!HAS_S) {
#pragma unroll
            for (int pp = 0; pp < NPAIR; ++pp) {
                exps(pp);
                round_sum(pp);
            }
        }
        // causal / ragged-end bound for tile t+1 (MASK_NEXT)
        const int room = (CAUSAL ? min(Skv - 1, qrow + diag) : Skv - 1) - (t + 1) * BN - 16 * hh;
        if (HAS_S) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) s_nxt[kb][r] = 0.f;
        }
        __builtin_amdgcn_sched_barrier(0);
        // Operand ring: slot i consumes fr[i % PF] and then refills the entry
        // slot i - 1 consumed (an MFMA still reading its operands must not see
        // them overwritten), so operands arrive PF - 1 slots early.  Each slot
        // is its own scheduling region (sched_barrier), and an empty asm that
        // reads and writes the running max (and sums) keeps the pure arithmetic
        // of the slot from drifting to the end of the tile.
        bf16x8 fr[PF];
        static_for<0, PF - 1>([&](auto ic) __attribute__((always_inline)) {
            fr[decltype(ic)::value] = fetch(decltype(ic)::value);
        });
        static_for<0, NM>([&](auto ic) __attribute__((always_inline)) {
            constexpr int i = decltype(ic)::value;
            const bf16x8 a = fr[i % PF];
            if constexpr (i + PF - 1 < NM) fr[(i + PF - 1) % PF] = fetch(i + PF - 1);
            if constexpr (i < NS) {
                constexpr int ks = i / KB, kb = i % KB;
                s_nxt[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s_nxt[kb], 0, 0, 0);
            } else {
                constexpr int j = i - NS, kb = j / (2 * CB), h2 = (j / CB) % 2, cb = j % CB;
                oacc[cb] =
                    __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[kb][h2], oacc[cb], 0, 0, 0);
                // the step's row sums right behind its first PV MFMA (same B)
                if constexpr (cb == 0) row_sum(pb[kb][h2]);
            }
            if constexpr (HAS_S) {
                static_for<0, NPAIR>([&](auto pc) __attribute__((always_inline)) {
                    constexpr int pp = decltype(pc)::value;
                    if constexpr (pp * EXP_SLOTS / NPAIR == i) exps(pp);
                    if constexpr (pp * EXP_SLOTS / NPAIR + LAG == i) round_sum(pp);
                });
                static_for<0, NMAXV>([&](auto vc) __attribute__((always_inline)) {
                    constexpr int v = decltype(vc)::value;
                    if constexpr (MAX0 + v * (NM - MAX0) / NMAXV == i) {
                        if (MASK_NEXT && (v / 16) * 32 + v % 16 > room)
                            s_nxt[v / 16][v % 16] = -INFINITY;
                        // (no quieting of NaNs: the scores are finite or
                        // -inf, and two maxima fold into one v_maximum3; the
                        // four-wave 64-key kernel keeps fmaxf, with which it
                        // does not spill)
                        if constexpr (NW == 8)
                            mx = __builtin_elementwise_maximum(mx, s_nxt[v / 16][v % 16]);
                        else
                            mx = fmaxf(mx, s_nxt[v / 16][v % 16]);
                    }
                });
            }
            if constexpr (HAS_S && MSUM) asm volatile("" : "+v"(mx));
            if constexpr (HAS_S && !MSUM) asm volatile("" : "+v"(rs0), "+v"(rs1), "+v"(mx));
            __builtin_amdgcn_sched_barrier(0);
        });
        if constexpr (!MSUM) l_i += rs0 + rs1;
        return HAS_S ? half_swap_max(mx) : -INFINITY;
    };

    // ---- main loop over K/V tiles ------------------------------------------
    // Every schedule runs its tiles in two loops: first the tiles that need no
    // mask, then the masked ones (compile-time tag), so the masking code never
    // sits in the common loop body.
    auto two_loops = [&](int t0, auto&& step) __attribute__((always_inline)) {
        int t = t0;
        const int split = max(t0, min(first_masked, n_tiles));
        for (; t < split; ++t) step(t, std::false_type{});
        for (; t < n_tiles; ++t) step(t, std::true_type{});
    };
    if (PIPE == 0) {
        two_loops(0, [&](int t, auto mask_tag) {
            dma(t, KS0, t, VS0);
            tile_barrier();
            if (wave_active(t)) {
                f32x16 s[KB];
                bf16x8 pb[KB][2];
                scores(kslot0, s);
                probs(s, softmax_stats(s, t, mask_tag), pb);
                pv(vslot0, pb);
            }
            tile_barrier();
        });
    } else if (PIPE == 1) {
        // tile t+1 streams into the other slot while tile t is computed from
        // LDS; one barrier per tile
        dma(0, KS0, 0, VS0);
        tile_barrier();
        two_loops(0, [&](int t, auto mask_tag) {
            const bool odd = t & 1;
            if (t + 1 < n_tiles) dma(t + 1, odd ? KS0 : KS1, t + 1, odd ? VS0 : VS1);
            if (wave_active(t)) {
                f32x16 s[KB];
                bf16x8 pb[KB][2];
                scores(odd ? kslot1 : kslot0, s);
                probs(s, softmax_stats(s, t, mask_tag), pb);
                pv(odd ? vslot1 : vslot0, pb);
            }
            tile_barrier();
        });
    } else if (PIPE == 2) {
        // Ping-pong.  LDS holds K_t, K_{t+1} and V_{t-1}, V_t in two-slot
        // rings (tile t in slot t&1).  Per tile t:
        //   phase 1: A: PV(t-1), S(t)          B: softmax(t)
        //   phase 2: A: softmax(t)             B: PV(t), S(t+1)
        // The global loads of K_{t+2} and V_{t+1} are issued at the start of
        // phase 1 and written to LDS at the end of phase 2 (into the slots of
        // K_t and V_{t-1}, whose last readers finished in phase 1).
        u32x4 kr[CH], vr[CH];  // tile data staged through registers
        // from the thread id, not the scalar wave index: the two groups' bodies
        // then stay exec-masked regions, which the register allocator handles
        // far better here than two scalar branches
        const bool group_b = (tid >> 6) >= 4;
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
        tile_barrier();
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
            tile_barrier();
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
            tile_barrier();
        });
        if (pv_pending) pv(((n_tiles - 1) & 1) ? vslot1 : vslot0, pb);
    } else {
        // Software pipeline.  Iteration t issues the MFMAs of S(t+1) and PV(t)
        // and, between them in program order, the exponentials of tile t and
        // the row max of tile t+1: a wave issues in order, so an MFMA followed
        // by independent VALU instructions keeps the matrix core and the VALU
        // busy together.  While iteration t runs LDS holds K_{t+1} and V_t,
        // and K_{t+2} and V_{t+1} stream into the slots of K_t and V_{t-1}
        // (tile j lives in slot j & 1).
        // Scores alternate between two register sets (A for even tiles, B for
        // odd ones), so the loop runs two tiles per trip.
        f32x16 sA[KB], sB[KB];
        bf16x8 pb[KB][2];
        float mx_next = -INFINITY;  // row max of the next tile's scores
        dma(0, KS0, 0, VS0);
        if (n_tiles > 1) dma_k(1, KS1);
        tile_barrier();
        if (wave_active(0)) {
            scores(kslot0, sA);
            mx_next = first_masked <= 0 ? tile_max(sA, 0, std::true_type{})
                                        : tile_max(sA, 0, std::false_type{});
        }
        tile_barrier();  // slot 0 takes K_2 at the end of iteration 0

        // Iteration t of the loop: PV(t) and S(t+1), up to the tile before the
        // wave's last active one.  The last active tile runs once after the
        // loop, without scores of a next tile (which would never be used: on
        // the last tile they would come from a stale K slot, on a causal
        // wave's last tile from keys past its diagonal); a wave then issues
        // only the loads and barriers of the tiles past its diagonal.  The
        // variant without S(t+1) sits outside the loop: inside it, the two
        // bodies together spilled.
        auto iter = [&](int t, f32x16 (&s_cur)[KB], f32x16 (&s_nxt)[KB], auto mask_tag) __attribute__((always_inline)) {
            const bool odd = t & 1;
            dma(t + 2 < n_tiles ? t + 2 : -1, odd ? KS1 : KS0,
                t + 1 < n_tiles ? t + 1 : -1, odd ? VS0 : VS1);
            const uint16_t* const k_next = odd ? kslot0 : kslot1;  // K_{t+1}
            const uint16_t* const v_cur = odd ? vslot1 : vslot0;   // V_t
            if (wave_active(t)) {
                const float m_ref = update_ref(mx_next);
                mx_next = fused_tile(k_next, v_cur, s_cur, s_nxt, pb, t, m_ref, std::true_type{},
                                     mask_tag);
            }
            tile_barrier();
        };
        // Two loops, one per masking mode of the next tile, each running two
        // tiles per trip (score sets A and B alternate).  The second loop, and
        // the last active tile, start with the current scores in set A.
        const int t_last = CAUSAL ? min(n_tiles - 1, (q_wave0 + 31 + diag) / BN) : n_tiles - 1;
        const int split = max(0, min(first_masked - 1, t_last));
        auto run = [&](int t0, int t1, auto mask_tag) __attribute__((always_inline)) {
            for (int t = t0; t < t1; t += 2) {
                iter(t, sA, sB, mask_tag);
                if (t + 1 < t1) iter(t + 1, sB, sA, mask_tag);
            }
        };
        run(0, split, std::false_type{});
        if (split & 1) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) sA[kb] = sB[kb];
        }
        run(split, t_last, std::true_type{});
        if ((t_last - split) & 1) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) sA[kb] = sB[kb];
        }
        {
            const int t = t_last;
            const bool odd = t & 1;
            dma(t + 2 < n_tiles ? t + 2 : -1, odd ? KS1 : KS0, t + 1 < n_tiles ? t + 1 : -1,
                odd ? VS0 : VS1);
            const float m_ref = update_ref(mx_next);
            fused_tile(odd ? kslot0 : kslot1, odd ? vslot1 : vslot0, sA, sB, pb, t, m_ref,
                       std::false_type{}, std::true_type{});
            tile_barrier();
        }
        for (int t = t_last + 1; t < n_tiles; ++t) {
            const bool odd = t & 1;
            dma(t + 2 < n_tiles ? t + 2 : -1, odd ? KS1 : KS0, t + 1 < n_tiles ? t + 1 : -1,
                odd ? VS0 : VS1);
            tile_barrier();
        }
    }

    // The next q-tile's Q is fetched before this one's output is stored, so
    // waiting for it does not wait for the stores (memory operations of a wave
    // complete in issue order).
    if (pass + 1 < n_pass) load_q(qt_of(pass + 1));
    __builtin_amdgcn_sched_barrier(0);

    // ---- epilogue: O = O^T / l, one query row per lane ----------------------
    // (fp32 or bf16 rows; optionally the row's log-sum-exp, natural log:
    // the reference m_i is in log2 units and includes the scale)
    // With split keys the row's unnormalised partials (m_i, l, O) go to the
    // workspace instead (the split combine normalises).
    const float l_row = MSUM ? lsum[0] : half_swap_sum(l_i);
    // (not with the ping-pong schedule, which has no registers to spare)
    const bool partial = PIPE != 2 && kv_splits > 1;
    const float inv = partial ? 1.f : 1.f / l_row;
    // The ping-pong schedule reads V once more after its last tile barrier.
    if (PIPE == 2) tile_barrier();
    // Output rows leave through LDS.  A lane holds runs of 4 consecutive
    // values of its row, so stores straight from registers touch 32 rows
    // (32 cache lines) per instruction.  Instead each wave writes one 128-byte
    // piece of each of its 32 rows (32 columns in fp32, 64 in bf16) into its
    // own staging region and reads it back so that 8 lanes hold the piece of
    // one row: each store instruction then writes 8 whole 128-byte lines.
    // Every wave has passed the final tile barrier, so no wave reads the K/V
    // slots any more and the staging regions may overlay them; within a wave
    // the LDS writes and reads complete in order.
    // The epilogue's kernel arguments are read here, behind an opaque zero
    // offset, instead of being held in scalar registers through the tile
    // loop, which is short of them.
    int kz;
    asm volatile("s_mov_b32 %0, 0" : "=s"(kz));
    const FwdArgs& ea = *reinterpret_cast<const FwdArgs*>(reinterpret_cast<const char*>(&args) + kz);
    const bool out16 = ea.out_bf16 && !partial;
    // lane-derived addresses are recomputed here from an opaque copy of the
    // lane index, rather than shared with values computed before the tile
    // loop (which would then stay live, in registers, through the loop)
    int elane = lane;
    asm volatile("" : "+v"(elane));
    const int el32 = elane & 31, ehh = elane >> 5;
    uint8_t* const stage = reinterpret_cast<uint8_t*>(lds) + wave * kFwdStageWaveBytes;
    constexpr int SROW = kFwdStageRowBytes;
    const long long row0 = (long long)bh * Sq + q_wave0;  // this wave's first row
    char* const obase = partial ? reinterpret_cast<char*>(ea.ws_o) : static_cast<char*>(ea.o);
    const int row_bytes = out16 ? 2 * D : 4 * D;
    // (all four LDS reads first: the stores go through generic pointers,
    // which the compiler would otherwise keep behind each read in turn)
    auto emit = [&](int piece) __attribute__((always_inline)) {
        u32x4 w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[j] = *reinterpret_cast<const u32x4*>(stage + ((elane >> 3) + 8 * j) * SROW +
                                                   (elane & 7) * 16);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = (elane >> 3) + 8 * j;
            if (q_wave0 + r < Sq) {
                const long long orow = partial ? (row0 + r) * kv_splits + split : row0 + r;
                *reinterpret_cast<u32x4*>(obase + orow * row_bytes + piece * 128 + (elane & 7) * 16) = w[j];
            }
        }
    };
    if (out16) {
        static_for<0, CB / 2>([&](auto pc) __attribute__((always_inline)) {
            constexpr int piece = decltype(pc)::value;
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x16& a = oacc[2 * piece + half];
                    const bf16x2 lo = {(__bf16)(a[4 * g] * inv), (__bf16)(a[4 * g + 1] * inv)};
                    const bf16x2 hi = {(__bf16)(a[4 * g + 2] * inv), (__bf16)(a[4 * g + 3] * inv)};
                    *reinterpret_cast<uint32_t*>(stage + el32 * SROW + (half * 32 + 8 * g + 4 * ehh) * 2) =
                        __builtin_bit_cast(uint32_t, lo);
                    *reinterpret_cast<uint32_t*>(stage + el32 * SROW + (half * 32 + 8 * g + 4 * ehh) * 2 + 4) =
                        __builtin_bit_cast(uint32_t, hi);
                }
            asm volatile("" ::: "memory");  // staging writes before the reads
            emit(piece);
            asm volatile("" ::: "memory");  // and the reads before the next piece's writes
        });
    } else {
        static_for<0, CB>([&](auto pc) __attribute__((always_inline)) {
            constexpr int cb = decltype(pc)::value;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 val = {oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv,
                                    oacc[cb][4 * g + 2] * inv, oacc[cb][4 * g + 3] * inv};
                *reinterpret_cast<u32x4*>(stage + el32 * SROW + (8 * g + 4 * ehh) * 4) =
                    __builtin_bit_cast(u32x4, val);
            }
            asm volatile("" ::: "memory");
            emit(cb);
            asm volatile("" ::: "memory");
        });
    }
    if (qrow < Sq && hh == 0) {
        const long long prow = ((long long)bh * Sq + qrow) * kv_splits + split;  // row if unsplit
        float* const mdst = partial ? ea.ws_m : ea.lse;
        if (mdst) mdst[prow] = partial ? m_i : (m_i + __builtin_log2f(l_row)) * kLn2;
        if (partial) ea.ws_l[prow] = l_row;
    }
    // Before the next q-tile's tile loads overwrite the staging regions, every
    // wave has read its own back (the stores already hold the data, so only
    // LDS operations are waited for, not the stores).
    if (pass + 1 < n_pass) asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }  // pass
}

}  // namespace attn
