// bf16 matrix multiplication C = A B for gfx950 (the paper's GEMM workload,
// Evaluation), fp32 accumulation, fp32 or bf16 output.
//
// Tiling.  A workgroup computes one BM x BN tile of C, streaming K in steps
// of BK through LDS.  Its WM x WN waves each own an (MB*32) x (NB*32)
// sub-tile: MB blocks of 32 rows of C by NB blocks of 32 columns, one
// v_mfma_f32_32x32x16_bf16 accumulator (16 fp32 per lane) per block pair.
//
// Orientation.  Each MFMA computes a transposed block, C^T = B^T A^T over 16
// values of k: the A operand is 32 columns of B (n) by 16 k, the B operand
// 16 k by 32 rows of A (m).  The accumulator then holds one row m of C per
// lane (lane & 31) and, in register r of lane half h, column
// 8*(r/4) + 4*h + r%4: four consecutive columns per register group, stored
// as one 16-byte (fp32) or 8-byte (bf16) write.
//
// Operands from LDS.  A tiles are [BM][BK+8] bf16 (rows padded by 16 bytes:
// consecutive rows start 4 banks apart, 16 lanes of a ds_read_b128 cover all
// 64 banks); lane (m, h) reads the 8 values k = 16*s + 8*h .. +7 of its row.
// B stored [N][K] is staged the same way ([BN][BK+8]).  B stored [K][N] is
// staged row-major ([BK][BN+32]) and its operand fetched with two
// ds_read_b64_tr_b16, which hand lane (n, h) the 8 values of column n at
// k = 16*s + 8*h .. +7: inside each 16-lane group, lane i addresses 4
// consecutive bf16 of row k0 + i/4 at column c0 + 4*(i%4), and lane j
// receives column c0 + j of rows k0 .. k0+3.
//
// Tile loads go straight from global memory into LDS (buffer loads with the
// LDS bit): a wave instruction writes 64 consecutive 16-byte chunks, so each
// lane's source address encodes the chunk's row, column and the padding
// (padding chunks re-read a valid chunk and are never used).  Rows past M
// (or N) and columns past N re-read the last valid row or chunk (their
// outputs are not stored), so no address leaves the operands; chunks past K
// get an offset past the buffer and come back as 0, so the ragged end of K
// adds exact zeros.
//
// Pipelining (the pipe knob of the latency model): PIPE 0 uses one LDS slot
// per operand (load, barrier, compute, barrier); PIPE 1 two slots, the next
// k-tile streaming in while the current one is multiplied; PIPE 2 three
// slots, two k-tiles in flight.  One barrier per k-tile; the loads are
// issued from inline assembly and waited for explicitly (lds_dma.h), so a
// slot's reads never wait for loads into another slot.
//
// Workgroup order.  The hardware deals workgroup ids round-robin to the 8
// XCDs; each XCD is given a contiguous range of logical tiles, and logical
// tiles run down groups of GM tile rows before moving right, so the tiles
// resident on one XCD share A row panels and B column panels in its L2.
//
// Two kernels share the loads, the operand layout and the epilogue: the
// generic one (every tile, the compiler scheduling each k-tile's MFMAs) and
// a hand-scheduled one for 256 x 256 tiles on four waves with
// v_mfma_f32_16x16x32_bf16 (gemm_sched_kernel, below), the large GEMMs' tile.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "common.h"
#include "lds_dma.h"

namespace attn {

namespace {

typedef __bf16 g_bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 g_bf16x2 __attribute__((ext_vector_type(2)));
typedef float g_f32x16 __attribute__((ext_vector_type(16)));
typedef short g_s16x4 __attribute__((ext_vector_type(4)));
typedef short g_s16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t g_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGroupM = 8;  // tile rows per group of the workgroup order

__device__ __forceinline__ g_s16x4 tr_read(const uint16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) g_s16x4*)(p));
}

template <int BM, int BN, int BK, bool B_NK>
struct GemmLds {
    static constexpr int A_STRIDE = BK + 8;                       // bf16 per A row
    static constexpr int B_ROWS = B_NK ? BN : BK;
    static constexpr int B_STRIDE = B_NK ? BK + 8 : BN + 32;      // bf16 per B row
    static constexpr int A_TILE = BM * A_STRIDE;
    static constexpr int B_TILE = B_ROWS * B_STRIDE;
    static constexpr int A_CPR = A_STRIDE / 8;                    // 16-byte chunks per row
    static constexpr int B_CPR = B_STRIDE / 8;
    static constexpr int A_REAL = BK / 8;                         // chunks holding data
    static constexpr int B_REAL = (B_NK ? BK : BN) / 8;
    static constexpr int A_PIECES = A_TILE / 512;                 // 64 chunks per piece
    static constexpr int B_PIECES = B_TILE / 512;
    static_assert(A_TILE % 512 == 0 && B_TILE % 512 == 0, "whole wave loads per tile");
};

// Tile of C (and K split) computed by this workgroup: the hardware deals
// workgroup ids round-robin to the XCDs; each XCD takes a contiguous range of
// logical indices, split-major (so an XCD's tiles share one K range of the
// panels), whose tiles run down groups of kGroupM tile rows before moving
// right.
struct GemmOrigin {
    int m0, n0, split;
};
__device__ __forceinline__ GemmOrigin gemm_origin(const GemmArgs& args, int BM, int BN) {
    const int n_wg = args.n_wg, num_xcds = args.num_xcds;
    const int wg = blockIdx.x;
    const int per = n_wg / num_xcds, rem = n_wg % num_xcds;
    const int xcd = wg % num_xcds, slot_id = wg / num_xcds;
    const int index =
        (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot_id;
    const int tiles_m = args.tiles_m, tiles_n = args.tiles_n;
    const int split = index / (tiles_m * tiles_n);
    const int logical = index - split * (tiles_m * tiles_n);
    const int group = logical / (kGroupM * tiles_n);
    const int first_m = group * kGroupM;
    const int gsize = min(tiles_m - first_m, kGroupM);
    const int in_group = logical - group * kGroupM * tiles_n;
    const int tm = first_m + in_group % gsize;
    const int tn = in_group / gsize;
    return {tm * BM, tn * BN, split};
}

// Direct-to-LDS loads of the k-tiles.  A k-tile's A and B regions are cut
// into pieces of 64 16-byte chunks (one wave instruction each); piece p goes
// to wave p % NW, A pieces first.  off[j] is the byte offset of this lane's
// source chunk for the wave's j-th piece relative to the k-tile's first
// element; the tile's own offset is a scalar.  Chunks past K (on the ragged
// last k-tile only, flagged per piece in this lane's `past_k` bits) read
// from an offset past the buffer and land as zeros.  SHIFT_B (B stored
// [K][N]): the rows of odd 8-row blocks of k hold their data 16 columns to
// the right inside the row padding (see the hand-scheduled kernel's reads).
template <int BM, int BN, int BK, int NW, bool B_NK, bool SHIFT_B = false>
struct GemmLoader {
    using L = GemmLds<BM, BN, BK, B_NK>;
    static constexpr int NP = L::A_PIECES + L::B_PIECES;
    static constexpr int NJ = (NP + NW - 1) / NW;  // pieces per wave (at most)
    static constexpr int NJ_MIN = NP / NW;         // pieces per wave (at least)
    static constexpr int SLOT = L::A_TILE + L::B_TILE;  // bf16 per LDS slot
    static constexpr int OOB = 0x7fffffff;  // any offset past the buffer reads zeros
    static_assert(NJ <= 32, "one bit per piece");

    dma_rsrc_t a_rsrc, b_rsrc;
    uint32_t lds0;
    int wave;
    // byte offsets of k-tile 0 in A and B, and per k-tile step
    uint32_t a_tile0, b_tile0, b_tile_step;
    int off[NJ];
    uint32_t past_k;

    // k0: the first k this workgroup multiplies (its K split's), a whole
    // number of k-tiles
    __device__ __forceinline__ GemmLoader(const GemmArgs& args, const uint16_t* lds, int wave_,
                                          int lane, int m0, int n0, int k0 = 0)
        : wave(wave_) {
        // with the wave index bounded, whether piece j is an A or a B piece,
        // or missing, folds at compile time wherever the counts allow
        __builtin_assume(wave >= 0 && wave < NW);
        const int M = args.M, N = args.N, K = args.K;
        a_rsrc = make_dma_rsrc(args.a, (uint32_t)((long long)M * K * 2));
        b_rsrc = make_dma_rsrc(args.b, (uint32_t)((long long)N * K * 2));
        lds0 = lds_address(lds);
        // 32-bit offsets: A and B are under 2 GiB each (checked on the host)
        a_tile0 = __builtin_amdgcn_readfirstlane(((uint32_t)m0 * (uint32_t)K + (uint32_t)k0) * 2u);
        b_tile0 = __builtin_amdgcn_readfirstlane(
            B_NK ? ((uint32_t)n0 * (uint32_t)K + (uint32_t)k0) * 2u
                 : ((uint32_t)k0 * (uint32_t)N + (uint32_t)n0) * 2u);
        b_tile_step = __builtin_amdgcn_readfirstlane(B_NK ? (uint32_t)BK * 2u
                                                          : (uint32_t)BK * (uint32_t)N * 2u);
        const int k_last = K - ((K + BK - 1) / BK - 1) * BK;  // k values of the last tile
        past_k = 0;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int piece = wave + j * NW;
            const int pos = (piece < L::A_PIECES ? piece : piece - L::A_PIECES) * 64 + lane;
            int o = 0, kc = 0;
            if (piece < L::A_PIECES) {
                const int r = pos / L::A_CPR, c = min(pos % L::A_CPR, L::A_REAL - 1);
                const int row = min(m0 + r, M - 1) - m0;
                o = (row * K + c * 8) * 2;
                kc = c * 8;
            } else if (B_NK) {
                const int r = pos / L::B_CPR, c = min(pos % L::B_CPR, L::B_REAL - 1);
                const int row = min(n0 + r, N - 1) - n0;
                o = (row * K + c * 8) * 2;
                kc = c * 8;
            } else {
                // columns past N (outputs never stored) re-read the last chunk of the
                // row, and so do the padding chunks
                const int r = pos / L::B_CPR;
                const int shift = SHIFT_B && ((r >> 3) & 1) ? 2 : 0;
                const int c = min(max(pos % L::B_CPR - shift, 0),
                                  min(L::B_REAL - 1, (N - n0) / 8 - 1));
                o = (r * N + c * 8) * 2;
                kc = r;
            }
            off[j] = o;
            past_k |= (kc >= k_last ? 1u : 0u) << j;
        }
    }

    // This wave's j-th piece of k-tile t into LDS slot s (nothing if the wave
    // has fewer pieces; the branch is wave-uniform).  LAST: t is the last
    // k-tile, whose chunks past K read zeros.
    template <bool LAST>
    __device__ __forceinline__ void piece(int t, int s, int j) const {
        __builtin_assume(wave >= 0 && wave < NW);
        const int p = wave + j * NW;
        if (p >= NP) return;
        const int o = LAST && ((past_k >> j) & 1u) ? OOB : off[j];
        const uint32_t dst = lds0 + (uint32_t)s * (SLOT * 2);
        if (p < L::A_PIECES)
            lds_dma16(a_rsrc, dst + p * 1024, o, a_tile0 + (uint32_t)t * (BK * 2));
        else
            lds_dma16(b_rsrc, dst + L::A_TILE * 2 + (p - L::A_PIECES) * 1024, o,
                      b_tile0 + (uint32_t)t * b_tile_step);
    }
    // all of this wave's pieces of k-tile t of n_k
    __device__ __forceinline__ void tile(int t, int s, int n_k) const {
        if (t == n_k - 1) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) piece<true>(t, s, j);
        } else {
#pragma unroll
            for (int j = 0; j < NJ; ++j) piece<false>(t, s, j);
        }
    }
};

// MFMA operands from an LDS slot: lane (row, h) of the A operand (16 k by 32
// rows of A) holds the 8 values k = 16*s + 8*h .. +7 of its row; the B
// operand likewise for a column of B (a row of B^T).
template <int BM, int BN, int BK, bool B_NK>
struct GemmFrags {
    using L = GemmLds<BM, BN, BK, B_NK>;
    int a_off, b_off;  // per-lane element offsets inside the slot's A and B tiles
    __device__ __forceinline__ GemmFrags(int lane, int wm0, int wn0) {
        const int l32 = lane & 31, hh = lane >> 5;
        a_off = (wm0 + l32) * L::A_STRIDE + hh * 8;
        if constexpr (B_NK) {
            b_off = (wn0 + l32) * L::B_STRIDE + hh * 8;
        } else {
            const int tr_row = (lane & 15) >> 2;
            const int tr_col = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
            b_off = (hh * 8 + tr_row) * L::B_STRIDE + wn0 + tr_col;
        }
    }
    __device__ __forceinline__ g_bf16x8 a(const uint16_t* slot, int mb, int s) const {
        return *reinterpret_cast<const g_bf16x8*>(slot + a_off + mb * 32 * L::A_STRIDE + s * 16);
    }
    __device__ __forceinline__ g_bf16x8 b(const uint16_t* slot, int nb, int s) const {
        const uint16_t* bt = slot + L::A_TILE;
        if constexpr (B_NK) {
            return *reinterpret_cast<const g_bf16x8*>(bt + b_off + nb * 32 * L::B_STRIDE + s * 16);
        } else {
            const uint16_t* p = bt + b_off + s * 16 * L::B_STRIDE + nb * 32;
            const g_s16x4 lo = tr_read(p);
            const g_s16x4 hi = tr_read(p + 4 * L::B_STRIDE);
            const g_s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            return __builtin_bit_cast(g_bf16x8, w);
        }
    }
};

// Epilogue through LDS: a lane holds 4-column runs of one row of each 32x32
// block, so storing from registers writes 16 (fp32) or 8 (bf16) bytes at
// each of 32 rows per instruction, which reach memory as partial lines.
// Each wave instead writes one piece of its 32 rows -- a block's 32 columns
// in fp32 (128 bytes), two blocks' 64 columns in bf16 -- into its own
// staging region (rows padded to 144 bytes, overlaying the k-tile slots,
// which no wave may still read: the caller has passed a barrier after its
// last LDS read), reads it back so that the lanes of one row hold its
// contiguous bytes, and stores whole lines.  The LDS writes and reads of a
// wave complete in order.  (mbase, nbase): the wave's sub-tile origin in C.
constexpr int kStageRow = 144;
template <int MB, int NB>
__device__ __forceinline__ void gemm_store(const g_f32x16 (&acc)[NB][MB], const GemmArgs& args,
                                           uint16_t* lds, int wave, int mbase, int nbase) {
    // lane-derived values recomputed from an opaque copy of the lane index
    // (not shared with values held through the k-loop)
    int elane = threadIdx.x & 63;
    asm volatile("" : "+v"(elane));
    const int el32 = elane & 31, ehh = elane >> 5;
    const int M = args.M, N = args.N;
    uint8_t* const stage = reinterpret_cast<uint8_t*>(lds) + wave * 32 * kStageRow;
    auto store_all = [&](auto bf16_tag) __attribute__((always_inline)) {
        constexpr bool BF16 = decltype(bf16_tag)::value;
        constexpr int ESZ = BF16 ? 2 : 4;
        constexpr int NBP = (BF16 && NB % 2 == 0) ? 2 : 1;  // 32-column blocks per piece
        constexpr int PB = 32 * NBP * ESZ;                  // bytes of a row's piece
        constexpr int LPR = PB / 16;                        // lanes per row on read-back
        constexpr int RPI = 64 / LPR;                       // rows per read instruction
        char* const cbase = static_cast<char*>(args.c);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
            for (int np = 0; np < NB / NBP; ++np) {
#pragma unroll
                for (int q = 0; q < NBP; ++q) {
                    const g_f32x16& c = acc[np * NBP + q][mb];
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        uint8_t* dst = stage + el32 * kStageRow + (q * 32 + 8 * g + 4 * ehh) * ESZ;
                        if constexpr (BF16) {
                            const g_bf16x2 lo = {(__bf16)c[4 * g], (__bf16)c[4 * g + 1]};
                            const g_bf16x2 hi = {(__bf16)c[4 * g + 2], (__bf16)c[4 * g + 3]};
                            *reinterpret_cast<uint32_t*>(dst) = __builtin_bit_cast(uint32_t, lo);
                            *reinterpret_cast<uint32_t*>(dst + 4) = __builtin_bit_cast(uint32_t, hi);
                        } else {
                            const float4 v = {c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
                            *reinterpret_cast<g_u32x4*>(dst) = __builtin_bit_cast(g_u32x4, v);
                        }
                    }
                }
                asm volatile("" ::: "memory");  // staging writes before the reads
                g_u32x4 w[32 / RPI];
#pragma unroll
                for (int j = 0; j < 32 / RPI; ++j)
                    w[j] = *reinterpret_cast<const g_u32x4*>(
                        stage + (elane / LPR + j * RPI) * kStageRow + (elane % LPR) * 16);
                const int col = nbase + np * NBP * 32 + (elane % LPR) * (16 / ESZ);
#pragma unroll
                for (int j = 0; j < 32 / RPI; ++j) {
                    const int row = mbase + mb * 32 + elane / LPR + j * RPI;
                    if (row < M && col < N)
                        *reinterpret_cast<g_u32x4*>(cbase + ((long long)row * N + col) * ESZ) = w[j];
                }
                asm volatile("" ::: "memory");  // and the reads before the next piece's writes
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    if (args.out_bf16)
        store_all(std::true_type{});
    else
        store_all(std::false_type{});
}

template <int BM, int BN, int BK, int WM, int WN, bool B_NK, int PIPE>
constexpr int gemm_waves_per_eu() {
    // one wave per SIMD when a wave holds 256 accumulators
    return (BM / (32 * WM)) * (BN / (32 * WN)) * 16 > 128 ? 1 : 2;
}

template <int BM, int BN, int BK, int WM, int WN, bool B_NK, int PIPE>
__global__ __launch_bounds__(WM * WN * 64, (gemm_waves_per_eu<BM, BN, BK, WM, WN, B_NK, PIPE>()))
void gemm_kernel(const GemmArgs args) {
    constexpr int NW = WM * WN;
    constexpr int MB = BM / (32 * WM);  // 32-row blocks of C per wave
    constexpr int NB = BN / (32 * WN);  // 32-column blocks of C per wave
    constexpr int KS = BK / 16;         // MFMA k-steps per k-tile
    constexpr int NSLOT = PIPE + 1;     // LDS slots: the load of k-tile t+PIPE overlaps t
    using Ld = GemmLoader<BM, BN, BK, NW, B_NK>;
    constexpr int SLOT = Ld::SLOT;
    static_assert(MB >= 1 && NB >= 1 && BK % 16 == 0, "tile shape");

    __shared__ __attribute__((aligned(16))) uint16_t lds[NSLOT * SLOT];

    const int K = args.K;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const GemmOrigin org = gemm_origin(args, BM, BN);
    const int wm0 = (wave % WM) * MB * 32, wn0 = (wave / WM) * NB * 32;
    const Ld ld(args, lds, wave, lane, org.m0, org.n0);
    const GemmFrags<BM, BN, BK, B_NK> fr(lane, wm0, wn0);

    g_f32x16 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[nb][mb][r] = 0.f;

    auto multiply = [&](int slot) __attribute__((always_inline)) {
        const uint16_t* const st = lds + slot * SLOT;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            g_bf16x8 af[MB], bf[NB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) af[mb] = fr.a(st, mb, ks);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bf[nb] = fr.b(st, nb, ks);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int mb = 0; mb < MB; ++mb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf[nb], af[mb],
                                                                          acc[nb][mb], 0, 0, 0);
        }
    };

    // Each barrier publishes the next k-tile (every wave first waits for its
    // own loads of it; loads complete in issue order) and certifies that all
    // waves have finished reading the slot the next load will overwrite.
    const int n_k = (K + BK - 1) / BK;
    if constexpr (PIPE == 0) {
        for (int t = 0; t < n_k; ++t) {
            ld.tile(t, 0, n_k);
            publish_barrier<0>();
            multiply(0);
            publish_barrier<0>();
        }
    } else if constexpr (PIPE == 1) {
        ld.tile(0, 0, n_k);
        publish_barrier<0>();
        for (int t = 0; t < n_k; ++t) {
            if (t + 1 < n_k) ld.tile(t + 1, (t + 1) & 1, n_k);
            multiply(t & 1);
            publish_barrier<0>();
        }
    } else {
        // three slots: k-tile t+2 streams in while t is multiplied and t+1
        // is complete or landing; a barrier waits only for t+1
        ld.tile(0, 0, n_k);
        if (n_k > 1) {
            ld.tile(1, 1, n_k);
            publish_barrier<Ld::NJ_MIN>();
        } else {
            publish_barrier<0>();
        }
        int s = 0;  // slot of k-tile t
        for (int t = 0; t < n_k; ++t) {
            const int s2 = s >= 1 ? s - 1 : 2;  // slot of k-tile t+2
            if (t + 2 < n_k) ld.tile(t + 2, s2, n_k);
            multiply(s);
            if (t + 2 < n_k)
                publish_barrier<Ld::NJ_MIN>();
            else
                publish_barrier<0>();
            s = s == 2 ? 0 : s + 1;
        }
    }
    static_assert(NSLOT * SLOT * 2 >= NW * 32 * kStageRow, "the staging regions fit the slots");
    gemm_store<MB, NB>(acc, args, lds, wave, org.m0 + wm0, org.n0 + wn0);
}

// The hand-scheduled kernel: four waves in a 2 x 2 grid over a 256 x 256
// tile, each owning 128 x 128 of C as 8 x 8 blocks of 16 x 16 (64
// accumulators of 4 registers, 256 in all): one wave per SIMD, so no other
// wave hides its latencies, and each operand fetched from LDS feeds eight
// MFMAs (0.5 KB of LDS reads per 32 K flops against 0.75 KB for the 128 x 64
// sub-tiles of eight waves).  It multiplies with v_mfma_f32_16x16x32_bf16,
// which at equal work and schedule ran at an 11% higher clock under the
// power limit than 32x32x16 (half the accumulator traffic per flop).
//
// Operands of a 32-k step: lane l of the MFMA's A operand holds column n =
// l % 16 of a 16-column block of B at k = 8 (l / 16) .. +7 (two transposed
// reads, or one 16-byte read when B is stored [N][K]), its B operand row m =
// l % 16 of a 16-row block of A at the same k (one 16-byte read); the
// accumulator then holds, in register r of lane l, C at row l % 16 and
// column 4 (l / 16) + r of the block.  In a transposed read, lanes 16..31
// address rows 8 below lanes 0..15; B rows are 144 banks apart (576 bytes),
// so those rows would fall on the same banks, and no linear padding keeps
// all eight rows of a read apart: the odd 8-row blocks of k are therefore
// stored 16 columns (8 banks) to the right inside the row padding.
//
// The k-loop is scheduled by hand at MFMA granularity: a step is 64 MFMAs
// (block (nb, mb) in slot 8 nb + mb), each slot its own scheduling region,
// and
//  - the operands of the next step are read in fixed slots of the current
//    one (kReadSlot16), well before their first use: the A blocks, used
//    throughout a step, into a second register set; B blocks 0..6 into the
//    registers of the current step's block three slots after its last MFMA
//    (one register set less); B block 7, last used at the end of the step,
//    into a second set;
//  - the barrier that publishes k-tile t+1 comes before the last step of
//    tile t (whose operands are already in registers), so that step reads
//    tile t+1, and it frees the slot of tile t for tile t+NSLOT: NSLOT - 1
//    k-tiles are in flight while one is multiplied.
// A CU's texture path moves about 64 bytes of LDS-bound load data per clock,
// so a k-tile's loads (one 1 KB instruction per piece) take about half as
// long to issue as its MFMAs: the pieces of tile u are spread evenly over
// the steps after the barrier that frees its slot -- with three or more
// slots over the tile's KS steps (phase p in the p-th of them: the last step
// of tile u-NSLOT, then steps 0 .. KS-2 of tile u-NSLOT+1), landing NSLOT-2
// tiles before they are read; with two slots over the first of those steps
// only, so the last of them still have a step to land.
// Each barrier waits only for the wave's own loads of the tile it publishes
// (vmcnt counts the loads of the NSLOT - 2 younger tiles, all issued in full
// before it).  K is a whole number of k-tiles (the planner's constraint), and
// the loads run on past the last tile: those tiles go to slots no tile needs
// any more and read zeros or unused data, never past the buffers, so every
// k-tile is the same code; the final barrier waits for them before the
// epilogue reuses the slots.
constexpr int kReadSlot16[16] = {10, 18, 26, 34, 42, 50, 58, 60,  // B blocks 0..7
                                 2, 4, 6, 8, 12, 14, 16, 20};     // A blocks 0..7

typedef float g_f32x4 __attribute__((ext_vector_type(4)));

// Epilogue of the 16 x 16 accumulator layout, staged in LDS in fp32 (written
// straight from the accumulator registers) for both output types: a piece
// is 32 rows by 64 columns (rows padded to 272 bytes); read back, each lane
// holds 16 contiguous bytes of a row of fp32 output, or 8 values that it
// rounds to bf16 (16 bytes).  The staging regions overlay the k-tile slots,
// which no wave may still read (the caller has passed a barrier after its
// last LDS read).  (mbase, nbase): the wave's sub-tile origin in C.
template <int MB16, int NB16>
__device__ __forceinline__ void gemm_store16(const g_f32x4 (&acc)[NB16][MB16], const GemmArgs& args,
                                             uint16_t* lds, int wave, int mbase, int nbase) {
    constexpr int ROW = 272;
    static_assert(MB16 % 2 == 0 && NB16 % 4 == 0, "pieces of 2 x 4 blocks");
    int elane = threadIdx.x & 63;
    asm volatile("" : "+v"(elane));
    const int M = args.M, N = args.N;
    uint8_t* const stage = reinterpret_cast<uint8_t*>(lds) + wave * 32 * ROW;
    char* const cbase = static_cast<char*>(args.c);
    const bool bf16 = args.out_bf16 != 0;
#pragma unroll
    for (int mp = 0; mp < MB16 / 2; ++mp) {
#pragma unroll
        for (int nq = 0; nq < NB16 / 4; ++nq) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    *reinterpret_cast<g_u32x4*>(stage + (16 * i + (elane & 15)) * ROW +
                                                (16 * j + 4 * (elane >> 4)) * 4) =
                        __builtin_bit_cast(g_u32x4, acc[nq * 4 + j][mp * 2 + i]);
            asm volatile("" ::: "memory");  // staging writes before the reads
            const int row0 = mbase + mp * 32;
            if (!bf16) {
                // 16 lanes per row, 4 rows per read
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int r = (elane >> 4) + 4 * q;
                    const g_u32x4 w =
                        *reinterpret_cast<const g_u32x4*>(stage + r * ROW + (elane & 15) * 16);
                    const int row = row0 + r, col = nbase + nq * 64 + (elane & 15) * 4;
                    if (row < M && col < N)
                        *reinterpret_cast<g_u32x4*>(cbase + ((long long)row * N + col) * 4) = w;
                }
            } else {
                // 8 lanes per row, 8 values each
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int r = (elane >> 3) + 8 * q;
                    const uint8_t* src = stage + r * ROW + (elane & 7) * 32;
                    const g_u32x4 lo = *reinterpret_cast<const g_u32x4*>(src);
                    const g_u32x4 hi = *reinterpret_cast<const g_u32x4*>(src + 16);
                    g_u32x4 packed;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        // elements into plain variables first: this compiler
                        // turns __builtin_bit_cast of a vector element
                        // expression into element 0
                        const g_u32x4& h = e < 2 ? lo : hi;
                        const uint32_t x0 = h[2 * (e % 2)], x1 = h[2 * (e % 2) + 1];
                        const g_bf16x2 pr = {(__bf16)__builtin_bit_cast(float, x0),
                                             (__bf16)__builtin_bit_cast(float, x1)};
                        packed[e] = __builtin_bit_cast(uint32_t, pr);
                    }
                    const int row = row0 + r, col = nbase + nq * 64 + (elane & 7) * 8;
                    if (row < M && col < N)
                        *reinterpret_cast<g_u32x4*>(cbase + ((long long)row * N + col) * 2) = packed;
                }
            }
            asm volatile("" ::: "memory");  // and the reads before the next piece's writes
            __builtin_amdgcn_sched_barrier(0);
        }
    }
}

// acc += a^T b on v_mfma_f32_16x16x32_bf16 with the accumulator held in the
// accumulator registers.  Through the compiler builtin this kernel's 64
// accumulators get the vector-register form and are shuffled between the two
// register files on every k-tile; the inline form pins them.  What the
// compiler would otherwise guard: the operands come from LDS reads, and its
// wait-count pass covers the asm's register operands like any other use; an
// accumulator is updated once per 64 MFMAs, never by back-to-back
// dependent ones; operand registers are rewritten only slots after their last
// MFMA (kReadSlot16); and the accumulators are read only after the k-loop,
// behind explicit wait states (mfma16_drain).
__device__ __forceinline__ void mfma16(g_f32x4& acc, const g_bf16x8& a, const g_bf16x8& b) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// wait states between the last MFMA and reads of its accumulators (more
// than a 16-pass MFMA needs)
__device__ __forceinline__ void mfma16_drain() { asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"); }

template <int BK, bool B_NK, int PIPE>
__global__ __launch_bounds__(256, 1) void gemm_sched_kernel(const GemmArgs args) {
    constexpr int BM = 256, BN = 256, NW = 4;
    constexpr int MB16 = 8, NB16 = 8;  // 16-row and 16-column blocks per wave
    constexpr int NSLOT = PIPE + 1;
    constexpr int KS = BK / 32;        // 32-k steps per k-tile
    constexpr int NM = MB16 * NB16;    // MFMA slots per step
    using Ld = GemmLoader<BM, BN, BK, NW, B_NK, !B_NK>;
    using L = GemmLds<BM, BN, BK, B_NK>;
    constexpr int SLOT = Ld::SLOT;
    static_assert(B_NK || BN + 16 <= L::B_STRIDE, "the shifted rows fit the padding");
    constexpr int PHASES = NSLOT >= 3 ? KS : 1;  // steps a tile's loads are spread over
    static_assert(NSLOT >= 2 && NSLOT <= 4, "two to four LDS slots");
    static_assert(KS == 1 || KS == 2, "k-tiles of 32 or 64");
    static_assert(2 * Ld::NJ < 64, "vmcnt holds 6 bits");

    __shared__ __attribute__((aligned(16))) uint16_t lds[NSLOT * SLOT];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const GemmOrigin org = gemm_origin(args, BM, BN);
    const int wm0 = (wave & 1) * 128, wn0 = (wave >> 1) * 128;
    // this workgroup's K range: its split's chunk (all of K unsplit)
    const int k0 = org.split * args.k_chunk;
    const int K = min(args.k_chunk, args.K - k0);
    const Ld ld(args, lds, wave, lane, org.m0, org.n0, k0);
    // per-lane element offsets of the operand reads inside a slot
    const int a_off = (wm0 + (lane & 15)) * L::A_STRIDE + 8 * (lane >> 4);
    const int b_off = B_NK ? L::A_TILE + (wn0 + (lane & 15)) * L::B_STRIDE + 8 * (lane >> 4)
                           : L::A_TILE + (8 * (lane >> 4) + ((lane & 15) >> 2)) * L::B_STRIDE +
                                 wn0 + 4 * (lane & 3) + 16 * ((lane >> 4) & 1);
    // waves below this index load NJ pieces per tile, the others NJ_MIN
    const bool more = wave < Ld::NP - Ld::NJ_MIN * NW;

    // Publish a k-tile once this wave's loads of it have landed, with its
    // loads of the NSLOT - 2 tiles issued after it still in flight.
    auto publish = [&]() __attribute__((always_inline)) {
        if (more)
            publish_barrier<(NSLOT - 2) * Ld::NJ>();
        else
            publish_barrier<(NSLOT - 2) * Ld::NJ_MIN>();
    };
    const int n_k = K / BK;

    g_f32x4 acc[NB16][MB16];
#pragma unroll
    for (int nb = 0; nb < NB16; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB16; ++mb) acc[nb][mb] = g_f32x4{0.f, 0.f, 0.f, 0.f};

    // operands: A blocks in two sets (parity of the step), B blocks 0..6 in
    // one, B block 7 in two
    g_bf16x8 opa[2][MB16], opb[NB16 - 1], opb7[2];
    // operand f of step ks from the slot at `slot` into the set of parity
    // par: B block f (f < 8), else A block f - 8
    auto read = [&](int par, int f, const uint16_t* slot, int ks) __attribute__((always_inline)) {
        if (f < NB16) {
            g_bf16x8 v;
            if constexpr (B_NK) {
                v = *reinterpret_cast<const g_bf16x8*>(slot + b_off + f * 16 * L::B_STRIDE + ks * 32);
            } else {
                const uint16_t* p = slot + b_off + ks * 32 * L::B_STRIDE + f * 16;
                const g_s16x4 lo = tr_read(p);
                const g_s16x4 hi = tr_read(p + 4 * L::B_STRIDE);
                const g_s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
                v = __builtin_bit_cast(g_bf16x8, w);
            }
            if (f < NB16 - 1)
                opb[f] = v;
            else
                opb7[par] = v;
        } else {
            opa[par][f - NB16] = *reinterpret_cast<const g_bf16x8*>(
                slot + a_off + (f - NB16) * 16 * L::A_STRIDE + ks * 32);
        }
    };

    // tiles 0 .. NSLOT-2, publish tile 0, then load phase 0 of tile NSLOT-1
    // (the steady state issues it in the last step of tile -1)
#pragma unroll
    for (int u = 0; u < NSLOT - 1; ++u)
#pragma unroll
        for (int j = 0; j < Ld::NJ; ++j) ld.template piece<false>(u, u, j);
    publish();
#pragma unroll
    for (int j = 0; j < Ld::NJ / PHASES; ++j) ld.template piece<false>(NSLOT - 1, NSLOT - 1, j);
#pragma unroll
    for (int f = 0; f < 16; ++f) read(0, f, lds, 0);

    // Step ks of k-tile t (slot s) with its operands in the sets of parity PAR.
    auto step = [&](int t, int s, auto ks_tag, auto par_tag) __attribute__((always_inline)) {
        constexpr int ks = decltype(ks_tag)::value;
        constexpr int PAR = decltype(par_tag)::value;
        constexpr bool LAST = ks == KS - 1;
        // this step's load phase: the first phase of tile t+NSLOT after the
        // barrier, else phase ks+1 of tile t+NSLOT-1
        constexpr int P = LAST ? 0 : ks + 1;
        constexpr int J0 = P < PHASES ? P * Ld::NJ / PHASES : 0;
        constexpr int J1 = P < PHASES ? (P + 1) * Ld::NJ / PHASES : 0;
        const int s_next = s + 1 == NSLOT ? 0 : s + 1;
        const int s_prev = s == 0 ? NSLOT - 1 : s - 1;  // slot of tile t-1, then t+NSLOT-1
        const int u = LAST ? t + NSLOT : t + NSLOT - 1;
        const int su = LAST ? s : s_prev;
        // the last step reads step 0 of tile t+1 (stale but harmless after
        // the last tile: never used)
        const uint16_t* const src = lds + (LAST ? s_next : s) * SLOT;
        constexpr int nks = LAST ? 0 : ks + 1;
        if constexpr (LAST) publish();
        static_for<0, NM>([&](auto ic) __attribute__((always_inline)) {
            constexpr int i = decltype(ic)::value;
            constexpr int nb = i / MB16, mb = i % MB16;
            mfma16(acc[nb][mb], nb < NB16 - 1 ? opb[nb] : opb7[PAR], opa[PAR][mb]);
            static_for<0, 16>([&](auto fc) __attribute__((always_inline)) {
                constexpr int f = decltype(fc)::value;
                if constexpr (kReadSlot16[f] == i) read(PAR ^ 1, f, src, nks);
            });
            static_for<J0, J1>([&](auto jc) __attribute__((always_inline)) {
                constexpr int j = decltype(jc)::value;
                if constexpr ((j - J0) * NM / (J1 - J0) == i) ld.template piece<false>(u, su, j);
            });
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    int t = 0, s = 0;  // k-tile and its slot
    auto advance = [&]() __attribute__((always_inline)) {
        s = s + 1 == NSLOT ? 0 : s + 1;
        ++t;
    };
    if constexpr (KS == 2) {
        for (; t < n_k; advance()) {
            step(t, s, I0{}, I0{});
            step(t, s, I1{}, I1{});
        }
    } else {
        // one step per tile: the register sets alternate per tile, two tiles
        // per iteration
        for (; t + 1 < n_k; advance()) {
            step(t, s, I0{}, I0{});
            advance();
            step(t, s, I0{}, I1{});
        }
        if (t < n_k) step(t, s, I0{}, I0{});
    }
    // every wave's reads (the last, unused ones included) have completed
    // before the staging regions overlay the slots
    publish_barrier<0>();
    mfma16_drain();
    static_assert(NSLOT * SLOT * 2 >= NW * 32 * 272, "the staging regions fit the slots");
    if (args.k_splits > 1) {
        // a split writes its fp32 partial tile to the workspace
        GemmArgs pa = args;
        pa.c = args.ws + (long long)org.split * args.M * args.N;
        pa.out_bf16 = 0;
        gemm_store16<MB16, NB16>(acc, pa, lds, wave, org.m0 + wm0, org.n0 + wn0);
    } else {
        gemm_store16<MB16, NB16>(acc, args, lds, wave, org.m0 + wm0, org.n0 + wn0);
    }
}

// C = the sum of the K-split partials ws[s] (fp32 [M][N]) in split order,
// four consecutive values per thread (M N is a multiple of 8, since N is);
// fp32 or bf16 (round to nearest even) output.
template <bool BF16>
__global__ __launch_bounds__(256) void gemm_split_sum(const float* __restrict__ ws,
                                                      void* __restrict__ c, long long mn,
                                                      int splits) {
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= mn / 4) return;
    g_f32x4 sum = __builtin_nontemporal_load(reinterpret_cast<const g_f32x4*>(ws) + i);
    for (int s = 1; s < splits; ++s)
        sum += __builtin_nontemporal_load(reinterpret_cast<const g_f32x4*>(ws + s * mn) + i);
    if constexpr (BF16) {
        const float x0 = sum[0], x1 = sum[1], x2 = sum[2], x3 = sum[3];
        const g_bf16x2 lo = {(__bf16)x0, (__bf16)x1}, hi = {(__bf16)x2, (__bf16)x3};
        const uint2 w = {__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi)};
        reinterpret_cast<uint2*>(c)[i] = w;
    } else {
        reinterpret_cast<g_f32x4*>(c)[i] = sum;
    }
}

template <int BM, int BN, int BK, bool B_NK, int PIPE>
constexpr bool gemm_lds_fits() {
    using L = GemmLds<BM, BN, BK, B_NK>;
    return (PIPE + 1) * (L::A_TILE + L::B_TILE) * 2 <= 160 * 1024;
}

// A compiled GEMM kernel: its entry point and workgroup size.
struct GemmKernel {
    const void* fn = nullptr;
    int threads = 0;
};

template <int BM, int BN, int BK, int WM, int WN, bool B_NK, int PIPE>
GemmKernel tile_kernel() {
    if constexpr (gemm_lds_fits<BM, BN, BK, B_NK, PIPE>())
        return {reinterpret_cast<const void*>(&gemm_kernel<BM, BN, BK, WM, WN, B_NK, PIPE>),
                WM * WN * 64};
    return {};
}

template <int BK, bool B_NK, int PIPE>
GemmKernel sched_kernel() {
    if constexpr (PIPE >= 1 && gemm_lds_fits<256, 256, BK, B_NK, PIPE>())
        return {reinterpret_cast<const void*>(&gemm_sched_kernel<BK, B_NK, PIPE>), 256};
    return {};
}

template <int BM, int BN, int BK, int WM, int WN, bool B_NK>
GemmKernel tile_kernel(int pipe) {
    switch (pipe) {
        case 0: return tile_kernel<BM, BN, BK, WM, WN, B_NK, 0>();
        case 1: return tile_kernel<BM, BN, BK, WM, WN, B_NK, 1>();
        case 2: return tile_kernel<BM, BN, BK, WM, WN, B_NK, 2>();
        default: return {};
    }
}

template <int BK, bool B_NK>
GemmKernel sched_kernel(int pipe) {
    switch (pipe) {
        case 1: return sched_kernel<BK, B_NK, 1>();
        case 2: return sched_kernel<BK, B_NK, 2>();
        case 3: return sched_kernel<BK, B_NK, 3>();
        default: return {};
    }
}

// The kernel a plan names: 256 x 256 tiles on four waves are the
// hand-scheduled kernel, every other tile the generic one.  No kernel (fn
// null) if that variant is not compiled or its LDS does not fit.
GemmKernel gemm_variant(const GemmPlan& p) {
#define ATTN_G(BM, BN, BK, WM, WN)                                                             \
    if (p.block_m == BM && p.block_n == BN && p.block_k == BK && p.waves_m == WM &&              \
        p.waves_n == WN)                                                                       \
        return p.b_nk ? tile_kernel<BM, BN, BK, WM, WN, true>(p.pipe)                          \
                      : tile_kernel<BM, BN, BK, WM, WN, false>(p.pipe);
    ATTN_G(64, 64, 64, 2, 2) ATTN_G(128, 128, 32, 2, 2) ATTN_G(128, 128, 64, 2, 2)
    ATTN_G(256, 128, 32, 2, 2) ATTN_G(256, 128, 64, 2, 2) ATTN_G(128, 256, 32, 2, 2)
    ATTN_G(128, 256, 64, 2, 2) ATTN_G(256, 256, 32, 2, 4) ATTN_G(256, 256, 64, 2, 4)
#undef ATTN_G
#define ATTN_SCHED(BK)                                                                       \
    if (gemm_hand_scheduled(p.block_m, p.block_n, p.waves_m, p.waves_n) && p.block_k == BK)    \
        return p.b_nk ? sched_kernel<BK, true>(p.pipe) : sched_kernel<BK, false>(p.pipe);
    ATTN_SCHED(32) ATTN_SCHED(64)
#undef ATTN_SCHED
    return {};
}

}  // namespace

hipError_t launch_gemm(const GemmPlan& p, const void* a, const void* b, void* c, int M, int N,
                       int K, int out_bf16, int num_xcds, float* workspace, hipStream_t stream) {
    const GemmKernel kern = gemm_variant(p);
    if (!kern.fn) return hipErrorInvalidValue;
    const bool sched = gemm_hand_scheduled(p.block_m, p.block_n, p.waves_m, p.waves_n);
    if (sched && K % p.block_k != 0) return hipErrorInvalidValue;
    const int splits = p.k_splits > 1 ? p.k_splits : 1;
    if (splits > 1 && (!sched || !workspace || p.k_chunk % p.block_k != 0 ||
                       (long long)(splits - 1) * p.k_chunk >= K ||
                       (long long)splits * p.k_chunk < K ||
                       p.grid != (long long)p.tiles_m * p.tiles_n * splits))
        return hipErrorInvalidValue;
    GemmArgs args;
    args.a = static_cast<const uint16_t*>(a);
    args.b = static_cast<const uint16_t*>(b);
    args.c = c;
    args.M = M;
    args.N = N;
    args.K = K;
    args.tiles_m = p.tiles_m;
    args.tiles_n = p.tiles_n;
    args.n_wg = (int)p.grid;
    args.num_xcds = num_xcds;
    args.out_bf16 = out_bf16;
    args.k_splits = splits;
    args.k_chunk = splits > 1 ? p.k_chunk : K;
    args.ws = workspace;
    void* kargs[] = {&args};
    hipError_t e =
        hipLaunchKernel(kern.fn, dim3((unsigned)p.grid), dim3(kern.threads), kargs, 0, stream);
    if (e != hipSuccess || splits == 1) return e;
    const long long mn = (long long)M * N;
    const unsigned blocks = (unsigned)((mn / 4 + 255) / 256);
    if (out_bf16)
        hipLaunchKernelGGL(gemm_split_sum<true>, dim3(blocks), dim3(256), 0, stream, workspace, c,
                           mn, splits);
    else
        hipLaunchKernelGGL(gemm_split_sum<false>, dim3(blocks), dim3(256), 0, stream, workspace,
                           c, mn, splits);
    return hipGetLastError();
}

bool gemm_resources(const GemmPlan& p, KernelRes* out) {
    const GemmKernel kern = gemm_variant(p);
    if (!kern.fn) return false;
    hipFuncAttributes at;
    if (hipFuncGetAttributes(&at, kern.fn) != hipSuccess) return false;
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kern.fn, kern.threads, 0) !=
        hipSuccess)
        return false;
    out->wg_per_cu = blocks;
    out->scratch_bytes = (int)at.localSizeBytes;
    out->vgprs = at.numRegs;
    return true;
}

}  // namespace attn
