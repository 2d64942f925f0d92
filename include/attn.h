/*
 * attn.h -- C ABI of libattn.so: tiled exact softmax attention on MI355X
 * (gfx950), prefill (FlashAttention forward) and split-KV Flash-Decode.
 *
 * The operation.  The paper evaluates two attention kernels (Evaluation,
 * Experimental Setup and the Flash Attention / Flash Decode paragraphs):
 * Flash Attention -- query-key scores, a softmax over them, then the
 * softmax-weighted sum of value rows -- and Flash Decode, its one-query
 * form, whose key axis is cut into pieces handled in parallel and then
 * merged: partial results are gathered, a softmax is taken across them and
 * the output is formed (HEG paragraph of the latency-modelling section).
 * Written out, for every batch b, head h and query row i:
 *     s_ij   = scale * sum_c q[b][h][i][c] * k[b][h][j][c]
 *     o[b][h][i][c] = sum_{j in A_i} exp(s_ij) v[b][h][j][c] / sum_{j in A_i} exp(s_ij)
 * with A_i = {0..Skv-1} (non-causal) or {j : j <= i + Skv - Sq} (causal,
 * aligned to the bottom-right corner of the score matrix).
 *
 * Conventions common to every call:
 *   - q, k, v, o are DEVICE pointers (e.g. torch.Tensor.data_ptr() of a
 *     CUDA/HIP tensor), contiguous, 16-byte aligned.  The caller owns them
 *     and keeps them alive until the stream has executed the work.
 *   - bf16 means IEEE bfloat16 bit patterns (uint16 storage).
 *   - All calls are asynchronous on the stream set by attn_set_stream()
 *     (per host thread; the default is the null stream).  They return after
 *     enqueueing and never synchronise; device faults surface at the
 *     caller's next synchronisation.
 *   - Arguments are validated on the host before anything is launched; on
 *     error nothing is launched and o is untouched.
 *   - Return codes: ATTN_OK (0) or a negative ATTN_E* code; the message of
 *     the last failing call on this host thread is in attn_last_error().
 *   - There is no CPU fallback: without a gfx950 device the compute calls
 *     return ATTN_EUNSUPPORTED or ATTN_EHIP.
 */
#ifndef ATTN_H
#define ATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ATTN_OK 0
#define ATTN_EINVAL (-1)       /* null or misaligned pointer, a dim <= 0, bad buffer length */
#define ATTN_EUNSUPPORTED (-2) /* d not in {64,128}, causal with Sq > Skv, one head's K or V over \
                                  2 GiB (prefill), device not gfx950 */
#define ATTN_EHIP (-3)         /* HIP runtime or launch error (message in attn_last_error) */
#define ATTN_ENOMEM (-4)       /* workspace allocation failed */

#define ATTN_KIND_FWD 0
#define ATTN_KIND_DECODE 1

/* attn_fwd_ex and attn_gemm flags */
#define ATTN_OUT_BF16 1        /* the output is bf16 (round to nearest even) instead of fp32 */
/* attn_gemm flag */
#define ATTN_GEMM_B_NK 2       /* B is stored [N][K] (B^T row-major) instead of [K][N] */

/*
 * Prefill attention (Flash Attention).
 *   q: bf16 [B][H][Sq][d]      k, v: bf16 [B][H][Skv][d]
 *   o: fp32 [B][H][Sq][d]      (caller-allocated, fully overwritten)
 *   scale: softmax scale applied to q.k (typically 1/sqrt(d)).
 *   causal: 0 = every key, 1 = key j allowed for row i iff j <= i + Skv - Sq.
 * Supported: d in {64, 128}; any B, H, Sq, Skv >= 1 (ragged tails are
 * handled); causal requires Sq <= Skv.  B*H*Sq*d and B*H*Skv*d must fit in
 * int64.  Work: QK^T and PV on bf16 MFMA with fp32 accumulation, online
 * softmax in fp32; the probabilities are rounded to bf16 before PV and the
 * normaliser sums the rounded values.
 */
int attn_fwd(const void* q, const void* k, const void* v, float* o, int B, int H, int Sq,
             int Skv, int d, float scale, int causal);

/*
 * Prefill with grouped-query heads, a bf16 or fp32 output and an optional
 * log-sum-exp (variants of attn_fwd; attn_fwd(...) is attn_fwd_ex(..., lse =
 * NULL, Hq = Hkv = H, flags = 0)).
 *   q: bf16 [B][Hq][Sq][d]   k, v: bf16 [B][Hkv][Skv][d]   Hkv divides Hq;
 *   query head h reads key/value head h / (Hq / Hkv) (Hkv = 1: multi-query).
 *   o: [B][Hq][Sq][d], fp32, or bf16 with ATTN_OUT_BF16 (caller-allocated).
 *   lse: NULL, or fp32 [B][Hq][Sq] (4-byte aligned) receiving each row's
 *   log-sum-exp of the scaled, masked scores in natural log,
 *   lse_i = log sum_j exp(scale q_i.k_j), so softmax weights are
 *   exp(s_ij - lse_i) -- what a caller needs to merge partial attention
 *   results (split-KV, ring attention).
 * Split keys: when the heads and q-tiles are too few to fill the device,
 * the planner may split each head's keys (non-causal only) into chunks
 * handled by separate workgroups, as Flash Decode splits its reduction
 * dimension; their partial results (row max, sum, unnormalised output) go
 * to the per-stream workspace described under attn_decode, and a combine
 * kernel on the same stream writes o and lse.  Such a call may allocate or
 * grow that workspace (ATTN_ENOMEM on failure); the result equals the
 * unsplit one up to fp32 rounding.  Up to 256 splits, as long as the split
 * grid stays within four rounds of the device's compute units (which bounds
 * the workspace to rows * splits * (d + 2) * 4 bytes, at most ~136 MB).
 * attn_get_plan reports the choice (KV_SPLITS, KV_CHUNK).
 * Errors as attn_fwd; EINVAL also for Hkv not dividing Hq, unknown flags or
 * a misaligned lse; EUNSUPPORTED if one head's K or V exceeds 2 GiB.
 */
int attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int Sq, int Skv, int d, float scale, int causal, int flags);

/*
 * Single-query attention with the KV sequence split across workgroups
 * (Flash Decode), then a log-sum-exp combine of the partial results (with a
 * single split the partial kernel writes o itself: the combine would be the
 * identity).
 *   q: bf16 [B][H][d]      k, v: bf16 [B][H][Skv][d]      o: fp32 [B][H][d]
 *   scale is fixed to (float)(1/sqrt(d)).
 *   n_splits <= 0: the planner chooses the split count from the device's
 *   compute-unit count and HBM model; otherwise it is clamped to [1, Skv]
 *   and the chunk is ceil(Skv / n_splits) keys (empty splits are never
 *   launched).  Every split count gives the same result up to fp32
 *   rounding.
 * Workspace: B*H*n*(d+2)*4 bytes of device memory that the library owns and
 * keeps per stream, reused by every later call on that stream (decode and
 * split-key prefill; stream order serialises them) until the process ends.
 * A call that needs more than the stream's current workspace allocates the
 * next power of two in stream order (hipMallocAsync) and releases the old
 * buffer in stream order (hipFreeAsync) behind the work already enqueued
 * on that stream; it never waits for the device.  ATTN_ENOMEM if that
 * allocation fails.  Host threads that share a stream are serialised from
 * the moment a call takes the workspace until its kernels are enqueued, so
 * a growth on one thread cannot release a buffer another thread's call is
 * about to use.  No call synchronises.
 */
int attn_decode(const void* q, const void* k, const void* v, float* o, int B, int H, int Skv,
                int d, int n_splits);

/*
 * Decode with grouped-query heads, an optional log-sum-exp and an optional
 * caller-provided workspace (attn_decode(...) is attn_decode_ex(..., lse =
 * NULL, Hq = Hkv = H, workspace = NULL)).
 *   q: bf16 [B][Hq][d]   k, v: bf16 [B][Hkv][Skv][d]   o: fp32 [B][Hq][d]
 *   Hkv divides Hq; query head h reads key/value head h / (Hq / Hkv).  The
 *   query heads of one key/value head (up to 8 per workgroup) are served
 *   by the same workgroups, which read each K/V row once for all of them.
 *   lse: NULL, or fp32 [B][Hq] receiving each row's natural-log
 *   log-sum-exp (as attn_fwd_ex).
 *   workspace: NULL (the library's per-stream workspace), or a 16-byte
 *   aligned device buffer of at least attn_decode_workspace_bytes(...)
 *   bytes that the caller keeps alive until the stream has passed this
 *   call; calls that share it must be ordered on one stream.  With a
 *   caller workspace the call allocates nothing.
 * Errors as attn_decode; EINVAL also for Hkv not dividing Hq, a misaligned
 * lse or workspace, or a workspace smaller than needed.
 */
int attn_decode_ex(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                   int Hq, int Hkv, int Skv, int d, int n_splits, void* workspace,
                   size_t workspace_bytes);

/*
 * Decode that allocates nothing, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same operation, arguments, plan and kernels as
 * attn_decode_ex with workspace = NULL, and the same result bit for bit;
 * the split partials go to a static device array of
 * ATTN_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs
 * on until the process ends (its address is looked up once per device, on
 * the first call made with that device current).
 *   Limit: B * Hq * n * (d + 2) * 4 bytes must fit in the scratch (n = the
 *   planned or requested split count, as attn_decode_workspace_bytes
 *   reports); a larger call fails with ATTN_ENOMEM before any launch.
 *   Concurrency: every call on one device shares that device's scratch, and
 *   it keeps the last call's partials.  Calls ordered on one stream are
 *   safe; calls that can overlap on one device (different streams, or host
 *   threads with no ordering between their streams) race on it.
 * Calls no allocation routine (no hipMalloc, hipFree or stream-ordered
 * allocation); asynchronous on the thread's stream; errors as
 * attn_decode_ex, plus ATTN_ENOMEM for a call over the limit and ATTN_EHIP
 * if the scratch address cannot be obtained.
 */
#define ATTN_NOALLOC_SCRATCH_BYTES (16u << 20)
int attn_decode_noalloc(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                        int Hq, int Hkv, int Skv, int d, int n_splits);

/* Bytes of decode workspace attn_decode_ex needs for this problem (plans
 * the call; needs the device), or a negative ATTN_E* code. */
long long attn_decode_workspace_bytes(int B, int Hq, int Hkv, int Skv, int d, int n_splits);

/* Set the HIP stream (hipStream_t, or NULL for the null stream) used by
 * this host thread's subsequent calls.  Returns ATTN_OK. */
int attn_set_stream(void* hip_stream);

/* The stream currently set for this host thread. */
void* attn_get_stream(void);

/* Message describing the last failing call on this host thread ("" if none).
 * The pointer stays valid until the next call on this thread. */
const char* attn_last_error(void);

/*
 * Architecture description used by the planner (cf. the paper's
 * architecture-description section: structural properties from the
 * specification, performance properties from microbenchmarks).
 */
typedef struct attn_device_desc {
    char arch[32];              /* e.g. "gfx950" */
    int num_cus;                /* compute units */
    int num_xcds;               /* accelerator complex dies (separate L2s) */
    int simds_per_cu;           /* 4 on CDNA */
    int wave_size;              /* 64 */
    int lds_bytes_per_cu;       /* local data share capacity */
    int vgprs_per_simd_lane;    /* unified VGPR+AGPR file per lane and SIMD */
    int max_waves_per_simd;     /* wave slots per SIMD */
    double clock_ghz;           /* peak engine clock */
    double mfma_bf16_flops_per_clk_cu; /* dense bf16 MFMA throughput */
    double valu_lanes_per_clk_simd;    /* fp32 VALU lanes per clock per SIMD */
    double trans_cycles_per_op;        /* SIMD cycles of one wave-wide v_exp_f32 */
    double lds_bytes_per_clk_cu;       /* LDS read bandwidth */
    double l2_bytes_per_clk_xcd;       /* L2 read bandwidth per XCD */
    double hbm_bytes_per_s;            /* sustained HBM read bandwidth */
    double hbm_latency_us;             /* loaded HBM latency (for bytes in flight) */
    double launch_us;                  /* kernel launch + drain overhead */
    /* Offline-calibrated prefill resource model (cycles at clock_ghz), fitted
     * once per architecture from the block-size ablation
     * (paper_2609_29219_amd/plan_ablation.py --fit); attn_measure_device()
     * leaves them unchanged. */
    double issue_cycles_per_score;     /* non-MFMA issue cycles of a wave per score */
    double valu_mfma_overlap;          /* share of that hidden behind another wave's MFMAs */
    double tile_sync_cycles;           /* per K/V tile: barrier and slot hand-off */
    double tile_latency_cycles;        /* K/V tile load latency exposed without prefetch */
} attn_device_desc;

/* Fill *out from the current HIP device (structural properties) and the
 * built-in gfx950 performance properties.  Without a usable device, fills
 * the MI355X specification values and returns ATTN_EHIP (out still valid). */
int attn_query_device(attn_device_desc* out);

/* Characterise the current device: fills the structural fields as
 * attn_query_device() does, then runs isolated microbenchmarks (MFMA, fp32
 * VALU, v_exp_f32, LDS read and HBM stream rates; about a second, allocates
 * and frees 2 GiB of device memory, synchronises the device) and stores the
 * measured performance properties in *out.  The planner's built-in gfx950
 * values were collected this way once; this call re-measures them. */
int attn_measure_device(attn_device_desc* out);

/*
 * Plan query: writes a one-line, human-readable plan -- the named tile
 * symbols (BLOCK_M, BLOCK_N, WAVES, PIPE, KV_SPLITS, KV_CHUNK for
 * ATTN_KIND_FWD; N_SPLITS, CHUNK, ... for ATTN_KIND_DECODE), the grid size,
 * the modelled time in us and the binding resource -- for the given problem
 * into buf (NUL-terminated, truncated to buflen).  This is the paper's
 * reporting of solved schedule symbols under the names the program gave
 * them (Symbolic MLIR subsection: symbols carry source-level labels, so the
 * chosen values can be reported back by name), with the latency the model
 * predicts (Eq. heg-optimization).  Returns the full length of the line (excluding the
 * NUL) or a negative ATTN_E* code.  Sq is ignored for decode.  desc may be
 * NULL (use attn_query_device()).  Host-only; launches nothing.
 */
int attn_get_plan(int kind, int B, int H, int Sq, int Skv, int d, int causal, int n_splits,
                  char* buf, int buflen);
int attn_get_plan_for(const attn_device_desc* desc, int kind, int B, int H, int Sq, int Skv,
                      int d, int causal, int n_splits, char* buf, int buflen);

/*
 * Matrix multiplication C = A B, the paper's GEMM workload (Evaluation,
 * Experimental Setup and the GEMM paragraph: the dense, compute-bound case
 * with heavy operand reuse), tiled by the same latency model.
 *   a: bf16 [M][K] row-major.
 *   b: bf16 [K][N] row-major, or with ATTN_GEMM_B_NK bf16 [N][K] row-major
 *      (c[m][n] = sum_k a[m][k] * b[n][k]).
 *   c: [M][N] row-major, fp32, or bf16 with ATTN_OUT_BF16 (caller-allocated,
 *      fully overwritten).
 * Work: bf16 MFMA products with fp32 accumulation (blocked summation order),
 * rounded once to the output type.  When the plan splits K (K_SPLITS > 1 in
 * attn_gemm_plan: few output tiles, long K), each split's fp32 partial goes
 * to the library's per-stream workspace (stream-ordered allocation, grown
 * as for decode) and a second kernel sums the partials in split order, so
 * the result is the same for every call with that plan.  Supported: M >= 1,
 * N and K multiples of 8 (16-byte rows), A and B each at most 2 GiB.
 * Asynchronous on the thread's stream.
 * Errors: EINVAL for null or misaligned pointers, dims <= 0 or unknown
 * flags; EUNSUPPORTED for N or K not a multiple of 8, operands over 2 GiB,
 * or a device that is not gfx950; ENOMEM if a split plan's workspace cannot
 * be allocated; EHIP for launch errors.
 */
int attn_gemm(const void* a, const void* b, void* c, int M, int N, int K, int flags);

/* GEMM plan query (host only): the named tile symbols BLOCK_M, BLOCK_N,
 * BLOCK_K, WAVES_M, WAVES_N, PIPE, K_SPLITS (with the k values per split),
 * the grid, the modelled time in us and the
 * binding resource, as one NUL-terminated line in buf (truncated to buflen).
 * desc NULL: this device's description and its compiled kernels' real
 * register/occupancy footprint.  Returns the full line length or a
 * negative ATTN_E* code (the same argument checks as attn_gemm). */
int attn_gemm_plan(const attn_device_desc* desc, int M, int N, int K, int flags, char* buf,
                   int buflen);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H */
