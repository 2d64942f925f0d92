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
    using L = GemmLds<BM, BN, BK, B_NK>;
    constexpr int NP = L::A_PIECES + L::B_PIECES;
    constexpr int NJ = (NP + NW - 1) / NW;  // pieces per wave (at most)
    constexpr int NJ_MIN = NP / NW;         // pieces per wave (at least)
    constexpr int SLOT = L::A_TILE + L::B_TILE;  // bf16 per slot
    static_assert(MB >= 1 && NB >= 1 && BK % 16 == 0, "tile shape");

    __shared__ __attribute__((aligned(16))) uint16_t lds[NSLOT * SLOT];

    const int M = args.M, N = args.N, K = args.K;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31;
    const int hh = lane >> 5;

    // ---- tile of this workgroup (XCD ranges, then groups of tile rows) ----
    const int n_wg = args.n_wg, num_xcds = args.num_xcds;
    const int wg = blockIdx.x;
    const int per = n_wg / num_xcds, rem = n_wg % num_xcds;
    const int xcd = wg % num_xcds, slot_id = wg / num_xcds;
    const int logical =
        (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + slot_id;
    const int tiles_m = args.tiles_m, tiles_n = args.tiles_n;
    const int group = logical / (kGroupM * tiles_n);
    const int first_m = group * kGroupM;
    const int gsize = min(tiles_m - first_m, kGroupM);
    const int in_group = logical - group * kGroupM * tiles_n;
    const int tm = first_m + in_group % gsize;
    const int tn = in_group / gsize;
    const int m0 = tm * BM, n0 = tn * BN;

    const int wm = wave % WM, wn = wave / WM;
    const int wm0 = wm * MB * 32, wn0 = wn * NB * 32;  // wave sub-tile inside the tile

    // ---- direct-to-LDS loads -------------------------------------------------
    const dma_rsrc_t a_rsrc = make_dma_rsrc(args.a, (uint32_t)((long long)M * K * 2));
    const dma_rsrc_t b_rsrc = make_dma_rsrc(args.b, (uint32_t)((long long)N * K * 2));
    const uint32_t lds0 = lds_address(lds);
    const int oob = 0x7fffffff;  // any offset past the buffer reads zeros
    // Piece p (0 <= p < NP) goes to wave p % NW: A pieces first, then B.
    // off[j]: byte offset of this lane's source chunk for the wave's j-th
    // piece, relative to the k-tile's first element (the tile-dependent part
    // is the scalar offset).  kof(j): the chunk's k offset inside the tile,
    // recomputed on the ragged last k-tile only.
    int off[NJ];
    auto pos_of = [&](int j) __attribute__((always_inline)) {
        const int piece = wave + j * NW;
        return (piece < L::A_PIECES ? piece : piece - L::A_PIECES) * 64 + lane;
    };
    auto kof = [&](int j) __attribute__((always_inline)) -> int {
        const int pos = pos_of(j);
        if (wave + j * NW < L::A_PIECES) return min(pos % L::A_CPR, L::A_REAL - 1) * 8;
        if (B_NK) return min(pos % L::B_CPR, L::B_REAL - 1) * 8;
        return pos / L::B_CPR;
    };
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int piece = wave + j * NW;
        const bool is_a = piece < L::A_PIECES;
        const int pos = pos_of(j);
        int o = 0;
        if (is_a) {
            const int r = pos / L::A_CPR, c = min(pos % L::A_CPR, L::A_REAL - 1);
            const int row = min(m0 + r, M - 1) - m0;
            o = (row * K + c * 8) * 2;
        } else if (B_NK) {
            const int r = pos / L::B_CPR, c = min(pos % L::B_CPR, L::B_REAL - 1);
            const int row = min(n0 + r, N - 1) - n0;
            o = (row * K + c * 8) * 2;
        } else {
            // columns past N (outputs never stored) re-read the last chunk of the row
            const int c = min(min(pos % L::B_CPR, L::B_REAL - 1), (N - n0) / 8 - 1);
            const int r = pos / L::B_CPR;
            o = (r * N + c * 8) * 2;
        }
        off[j] = o;
    }
    // Issue this wave's pieces of k-tile t into LDS slot s (NJ_MIN or NJ
    // loads; the branches are wave-uniform).
    auto dma = [&](int t, int s) __attribute__((always_inline)) {
        const uint32_t a_dst = lds0 + s * SLOT * 2;
        const uint32_t b_dst = a_dst + L::A_TILE * 2;
        const int k0 = t * BK;
        const bool ragged = k0 + BK > K;
        const int a_base = ((long long)m0 * K + k0) * 2;
        const int b_base = B_NK ? ((long long)n0 * K + k0) * 2 : ((long long)k0 * N + n0) * 2;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int piece = wave + j * NW;
            if (piece >= NP) continue;
            const bool is_a = piece < L::A_PIECES;
            const int o = (ragged && kof(j) >= K - k0) ? oob : off[j];
            if (is_a)
                lds_dma16(a_rsrc, a_dst + piece * 1024, o, a_base);
            else
                lds_dma16(b_rsrc, b_dst + (piece - L::A_PIECES) * 1024, o, b_base);
        }
    };

    // ---- operands from LDS ---------------------------------------------------
    const int tr_row = (lane & 15) >> 2;
    const int tr_col = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
    auto a_frag = [&](const uint16_t* at, int mb, int s) __attribute__((always_inline)) {
        return *reinterpret_cast<const g_bf16x8*>(at + (wm0 + mb * 32 + l32) * L::A_STRIDE +
                                                  s * 16 + hh * 8);
    };
    auto b_frag = [&](const uint16_t* bt, int nb, int s) __attribute__((always_inline)) {
        if constexpr (B_NK) {
            return *reinterpret_cast<const g_bf16x8*>(bt + (wn0 + nb * 32 + l32) * L::B_STRIDE +
                                                      s * 16 + hh * 8);
        } else {
            const uint16_t* p = bt + (s * 16 + hh * 8 + tr_row) * L::B_STRIDE + wn0 + nb * 32 +
                                tr_col;
            const g_s16x4 lo = tr_read(p);
            const g_s16x4 hi = tr_read(p + 4 * L::B_STRIDE);
            const g_s16x8 w = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
            return __builtin_bit_cast(g_bf16x8, w);
        }
    };

    g_f32x16 acc[NB][MB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[nb][mb][r] = 0.f;

    auto multiply = [&](int slot) __attribute__((always_inline)) {
        const uint16_t* const at = lds + slot * SLOT;
        const uint16_t* const bt = at + L::A_TILE;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            g_bf16x8 af[MB], bf[NB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) af[mb] = a_frag(at, mb, ks);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bf[nb] = b_frag(bt, nb, ks);
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
            dma(t, 0);
            publish_barrier<0>();
            multiply(0);
            publish_barrier<0>();
        }
    } else if constexpr (PIPE == 1) {
        dma(0, 0);
        publish_barrier<0>();
        for (int t = 0; t < n_k; ++t) {
            if (t + 1 < n_k) dma(t + 1, (t + 1) & 1);
            multiply(t & 1);
            publish_barrier<0>();
        }
    } else {
        // three slots: k-tile t+2 streams in while t is multiplied and t+1
        // is complete or landing; a barrier waits only for t+1
        dma(0, 0);
        if (n_k > 1) {
            dma(1, 1);
            publish_barrier<NJ_MIN>();
        } else {
            publish_barrier<0>();
        }
        int s = 0;  // slot of k-tile t
        for (int t = 0; t < n_k; ++t) {
            const int s2 = s >= 1 ? s - 1 : 2;  // slot of k-tile t+2
            if (t + 2 < n_k) dma(t + 2, s2);
            multiply(s);
            if (t + 2 < n_k)
                publish_barrier<NJ_MIN>();
            else
                publish_barrier<0>();
            s = s == 2 ? 0 : s + 1;
        }
    }

    // ---- epilogue through LDS: a lane holds 4-column runs of one row of each
    // 32x32 block, so storing from registers writes 16 (fp32) or 8 (bf16)
    // bytes at each of 32 rows per instruction, which reach memory as partial
    // lines.  Each wave instead writes one piece of its 32 rows -- a block's
    // 32 columns in fp32 (128 bytes), two blocks' 64 columns in bf16 -- into
    // its own staging region (rows padded to 144 bytes, overlaying the k-tile
    // slots, which no wave reads after the last barrier), reads it back so
    // that the lanes of one row hold its contiguous bytes, and stores whole
    // lines.  The LDS writes and reads of a wave complete in order.
    constexpr int SROW = 144;
    static_assert(NSLOT * SLOT * 2 >= NW * 32 * SROW, "the staging regions fit the slots");
    // lane-derived values recomputed from an opaque copy of the lane index
    // (not shared with values held through the k-loop)
    int elane = lane;
    asm volatile("" : "+v"(elane));
    const int el32 = elane & 31, ehh = elane >> 5;
    uint8_t* const stage = reinterpret_cast<uint8_t*>(lds) + wave * 32 * SROW;
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
                        uint8_t* dst = stage + el32 * SROW + (q * 32 + 8 * g + 4 * ehh) * ESZ;
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
                    w[j] = *reinterpret_cast<const g_u32x4*>(stage + (elane / LPR + j * RPI) * SROW +
                                                             (elane % LPR) * 16);
                const int col = n0 + wn0 + np * NBP * 32 + (elane % LPR) * (16 / ESZ);
#pragma unroll
                for (int j = 0; j < 32 / RPI; ++j) {
                    const int row = m0 + wm0 + mb * 32 + elane / LPR + j * RPI;
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

template <int BM, int BN, int BK, bool B_NK, int PIPE>
constexpr bool gemm_lds_fits() {
    using L = GemmLds<BM, BN, BK, B_NK>;
    return (PIPE + 1) * (L::A_TILE + L::B_TILE) * 2 <= 160 * 1024;
}

// The pipe settings of one tile whose LDS footprint fits.
template <int BM, int BN, int BK, int WM, int WN, bool B_NK, typename F>
bool run_pipe(int pipe, F& f) {
    if (pipe == 0) {
        f.template run<BM, BN, BK, WM, WN, B_NK, 0>();
        return true;
    }
    if (pipe == 1) {
        if constexpr (gemm_lds_fits<BM, BN, BK, B_NK, 1>()) {
            f.template run<BM, BN, BK, WM, WN, B_NK, 1>();
            return true;
        }
    }
    if (pipe == 2) {
        if constexpr (gemm_lds_fits<BM, BN, BK, B_NK, 2>()) {
            f.template run<BM, BN, BK, WM, WN, B_NK, 2>();
            return true;
        }
    }
    return false;
}

// Calls F::template run<BM, BN, BK, WM, WN, B_NK, PIPE>() for the variant the
// plan names; false if no such variant is compiled.
template <typename F>
bool with_gemm_variant(const GemmPlan& p, F& f) {
#define ATTN_G(BM, BN, BK, WM, WN)                                                             \
    if (p.block_m == BM && p.block_n == BN && p.block_k == BK && p.waves_m == WM &&              \
        p.waves_n == WN) {                                                                     \
        return p.b_nk ? run_pipe<BM, BN, BK, WM, WN, true>(p.pipe, f)                          \
                      : run_pipe<BM, BN, BK, WM, WN, false>(p.pipe, f);                        \
    }
    ATTN_G(64, 64, 64, 2, 2) ATTN_G(128, 128, 32, 2, 2) ATTN_G(128, 128, 64, 2, 2)
    ATTN_G(256, 128, 32, 2, 2) ATTN_G(256, 128, 64, 2, 2) ATTN_G(128, 256, 32, 2, 2)
    ATTN_G(128, 256, 64, 2, 2) ATTN_G(256, 256, 32, 2, 4) ATTN_G(256, 256, 64, 2, 4)
#undef ATTN_G
    return false;
}

struct GemmLaunch {
    const GemmPlan& p;
    const GemmArgs& a;
    hipStream_t st;
    hipError_t err = hipErrorInvalidValue;
    template <int BM, int BN, int BK, int WM, int WN, bool B_NK, int PIPE>
    void run() {
        hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, WM, WN, B_NK, PIPE>), dim3((unsigned)p.grid),
                           dim3(WM * WN * 64), 0, st, a);
        err = hipGetLastError();
    }
};

struct GemmResources {
    KernelRes* r;
    bool ok = false;
    template <int BM, int BN, int BK, int WM, int WN, bool B_NK, int PIPE>
    void run() {
        const void* fn = reinterpret_cast<const void*>(&gemm_kernel<BM, BN, BK, WM, WN, B_NK, PIPE>);
        hipFuncAttributes at;
        if (hipFuncGetAttributes(&at, fn) != hipSuccess) return;
        int blocks = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, WM * WN * 64, 0) !=
            hipSuccess)
            return;
        r->wg_per_cu = blocks;
        r->scratch_bytes = (int)at.localSizeBytes;
        r->vgprs = at.numRegs;
        ok = true;
    }
};

}  // namespace

hipError_t launch_gemm(const GemmPlan& p, const void* a, const void* b, void* c, int M, int N,
                       int K, int out_bf16, int num_xcds, hipStream_t stream) {
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
    GemmLaunch l{p, args, stream};
    if (!with_gemm_variant(p, l)) return hipErrorInvalidValue;
    return l.err;
}

bool gemm_resources(const GemmPlan& p, KernelRes* out) {
    GemmResources res{out};
    return with_gemm_variant(p, res) && res.ok;
}

}  // namespace attn
