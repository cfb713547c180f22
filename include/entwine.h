/*
 * entwine.h - C ABI of libentwine.so: one tensor-parallel rank's share of a
 * row-parallel GEMM-ReduceScatter on one MI355X (gfx950), with interleaved
 * tile production, per-tile ready flags and a concurrent tile reducer.
 *
 * Problem (paper Section 2.1 and Section 3.4, Equations 2-3): the local rank
 * holds A (M x K) and B (K x N), K being its slice of the reduction
 * dimension, and produces the M x N partial C = A B.  The output is split
 * into P equal row chunks; chunk d is rows [d M/P, (d+1) M/P).  The other P-1
 * ranks' partials are given as "peer" matrices Pi_q (q = 0 .. P-2, the ranks
 * other than the local one in ascending order), resident in device memory.
 * The reduced chunk is
 *     O_d = C[chunk d] + sum_q Pi_q[chunk d]      (peers added in order q).
 *
 * Element types: A, B, peers, partial and out are bfloat16 (raw 16-bit
 * words).  The GEMM accumulates in fp32 and stores the partial as bf16
 * (round to nearest even); the reducer sums in fp32 and rounds the output to
 * bf16 (nearest even).  All matrices are row-major with a leading dimension
 * in elements.
 *
 * Pointers: every matrix pointer is a DEVICE pointer on the context's device,
 * 16-byte aligned, with leading dimensions that are multiples of 8.  The
 * caller owns A, B, the peers, out and (when given) partial; they must stay
 * valid until the queued work completes.  The peer pointer array itself is a
 * HOST array, read during the call.  Streams are hipStream_t handles passed
 * as void* (NULL = the null stream).  Calls only enqueue work: they return
 * before the GPU finishes.  Errors are reported by return code only; the
 * message of the last failure is available from entwine_last_error().
 *
 * A context is not thread-safe; use one per (shape, stream pair).
 */
#ifndef ENTWINE_H
#define ENTWINE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ENTWINE_ABI_VERSION 3
#define ENTWINE_TILE 128      /* side of a reduction tile (Section 4.2) */
#define ENTWINE_MAX_P 8       /* chunk count supported (the paper's W <= 8) */
#define ENTWINE_DEST_ALL (-1) /* reduce every chunk (one-GPU emulation) */

typedef struct entwine_ctx entwine_ctx;

typedef enum {
  ENTWINE_OK = 0,
  ENTWINE_EINVAL = 1,      /* bad argument: shape, pointer, alignment, ld */
  ENTWINE_EUNSUPPORTED = 2,/* valid problem, but not for this config */
  ENTWINE_ENOMEM = 3,      /* device allocation failed */
  ENTWINE_EHIP = 4,        /* a HIP runtime call failed */
  ENTWINE_ETIMEOUT = 5     /* a reducer wait exceeded its bound (see query) */
} entwine_status;

/* Producer traversal orders (Section 3.1, Equation 1; Section 5.3.1). */
typedef enum {
  ENTWINE_ORDER_INTERLEAVED = 0, /* d = p mod P, l = p div P; l N-major in d */
  ENTWINE_ORDER_ROW_MAJOR = 1,   /* partition-contiguous, N fastest (Fig. 1 top) */
  ENTWINE_ORDER_M_MAJOR = 2      /* M fastest (producer default, ablation) */
} entwine_order;

/* Producer block (workgroup macro-tile) shapes, BM x BN; the reduction unit
 * stays 128 x 128 (Section 4.2), so a block covers (BM/128)(BN/128) tiles. */
typedef enum {
  ENTWINE_GEMM_256x256 = 0,
  ENTWINE_GEMM_256x128 = 1,
  ENTWINE_GEMM_128x256 = 2,
  ENTWINE_GEMM_128x128 = 3,
  ENTWINE_GEMM_NUM_CFGS = 4
} entwine_gemm_cfg;

/* Per-call configuration.  Zero / negative fields mean "default". */
typedef struct {
  int32_t order;          /* entwine_order (default INTERLEAVED) */
  int32_t gemm_cfg;       /* entwine_gemm_cfg, -1 = largest that divides */
  int32_t reduce_wgs;     /* x: reducer grid size, the communication budget
                             (Section 3.2); capped at the tile count and at
                             CUs - 1.  With DEST_ALL it is rounded up to a
                             multiple of P.  With launch 0, producers that
                             finish their blocks also take tiles, and -1
                             asks for no dedicated reducers at all (all CUs
                             produce, then reduce).  0 = default: none with
                             launch 0, 16 with launch 1, one per CU with
                             launch 2; the standalone reducer
                             (entwine_reduce_only and the sequential form)
                             then uses 16. */
  int32_t reduce_threads; /* b: threads per reducer workgroup, 128/256/512/1024
                             (0 = default = 1024) */
  int32_t timeout_us;     /* bound on one reducer wait, microseconds
                             (0 = 2 s); expiry sets ENTWINE_ETIMEOUT */
  int32_t withhold_peer;  /* test hook: peer q whose flags are not published
                             this call (-1 = none); forces a timeout */
  int32_t record_timing;  /* 1 = record events for entwine_last_timing() */
  int32_t group_m;        /* block order inside a partition: 1 = N-major (the
                             paper's), g > 1 = XCD-striped walk in groups of g
                             block rows (L2 reuse); 0 = default (4) */
  int32_t gemm_wgs;       /* producer workgroups (persistent; each takes
                             positions w, w + G, ...): 0 = default = the CUs,
                             minus x in the fused path, rounded down to a
                             multiple of 8 (one workgroup per CU) */
  int32_t launch;         /* fused path (distinct streams): 0 = one kernel
                             launch on gemm_stream whose first G workgroups
                             are producers and last x reducers of 256
                             threads (reduce_threads then does not apply;
                             G is capped so that all are resident);
                             1 = two kernels on the two streams (Section
                             4.3's form), with b threads per reducer;
                             2 = shared pool (Section 5.3.2): the producer
                             on every CU and x small reducer workgroups of
                             256 threads beside it (default x: one per CU);
                             1 and 0 partition the CUs instead */
  int32_t release_blocks; /* g: a producer workgroup publishes its finished
                             tiles after every g of its blocks, one release
                             each time (Section 5.3.2, release granularity:
                             every wave waits for its tile stores, plus an
                             L2 write-back with store_mode 1 or 2); 0 = default = 2; -1 = only once,
                             after its last block; release groups, where a
                             tile's flag waits for its whole group:
                             -2 = its row partition (chunk), -3 = the whole
                             output (the coarse end of Section 5.3.2's
                             ablation) */
  int32_t store_mode;     /* partial tile stores: 0 = write-through (a
                             release only waits for them), 1 = non-temporal,
                             2 = write-back (1 and 2 are written back from
                             L2 by each release) */
} entwine_config;

/* Fill *cfg with the defaults. */
void entwine_config_default(entwine_config* cfg);

/* Create a context for problems of shape (M, N, K, P) on `device`.  Owns the
 * per-tile flags, the epoch counter, a status word, timing events and, on
 * first need, an M x N bf16 partial scratch.  Requirements: 1 <= P <=
 * ENTWINE_MAX_P, M % (128 P) == 0, N % 128 == 0, K % 8 == 0, K > 0. */
entwine_status entwine_ctx_create(entwine_ctx** out, int32_t device, int64_t M, int64_t N,
                                  int64_t K, int32_t P);
entwine_status entwine_ctx_destroy(entwine_ctx* ctx);

/* The fused path (Sections 3.1-3.2, 4.1-4.3), enqueued after the prior work
 * on gemm_stream: the producer GEMM (tiles in cfg->order, a ready flag per
 * 128 x 128 tile), the synthetic peers' flag publication and the tile
 * reduction, concurrently.  With cfg->launch 0 (default) both roles are one
 * kernel launch on gemm_stream; with 1 and 2 the producer runs on
 * gemm_stream and the reducer on reduce_stream.  On return gemm_stream is
 * ordered after all of it.  When reduce_stream == gemm_stream the GEMM and
 * the reduction (two-stream kernels) run one after the other instead (the
 * unfused baseline).
 *   dest in [0, P): out is (M/P) x N, chunk dest (one rank's share);
 *   dest == ENTWINE_DEST_ALL: out is M x N, every chunk.
 *   peers: host array of P-1 device pointers, each an M x N matrix with
 *          leading dimension ldp; ignored when P == 1 (then out = bf16(A B)).
 *   partial: M x N bf16 workspace (ld ldc) receiving the local partial, or
 *          NULL for the context's own.
 * P == 1 reduces to a plain GEMM with a bf16 round trip. */
entwine_status entwine_gemm_rs(entwine_ctx* ctx, const void* A, int64_t lda, const void* B,
                               int64_t ldb, const void* const* peers, int64_t ldp, int32_t dest,
                               void* out, int64_t ldo, void* partial, int64_t ldc,
                               const entwine_config* cfg, void* gemm_stream, void* reduce_stream);

/* The fused path followed by the layer epilogue of the paper's layer-level
 * evaluation (Section 5.2: residual addition and RMSNorm after the
 * reduce-scatter), as one launch on `stream` (cfg->launch must be 0, else
 * ENTWINE_EUNSUPPORTED).  For every output row i of the destination
 * (rows as `out` of entwine_gemm_rs):
 *   h[i,:] = bf16(sum + residual[i,:])   the reduced row plus the residual,
 *                                        added in fp32 after the peers;
 *   y[i,:] = bf16(h[i,:] * (mean_j h[i,j]^2 + eps)^(-1/2) * gamma)
 *                                        from the stored bf16 h, fp32 math.
 * residual, h_out, y_out: bf16, out_rows x N (leading dimensions ldr, ldh,
 * ldy); gamma: bf16, N; eps > 0 and finite (ENTWINE_EINVAL otherwise);
 * N <= 16384 (a row is held in registers; ENTWINE_EUNSUPPORTED otherwise).
 * h_out may be the residual itself (same pointer and leading dimension: an
 * in-place update of the residual stream); otherwise h_out and y_out must
 * not overlap each other or any input.  Each row is
 * reduced and normalised by one workgroup once every tile of its tile row
 * is published, so both h and y are reproducible bit for bit.  Errors as
 * entwine_gemm_rs. */
entwine_status entwine_gemm_rs_rmsnorm(entwine_ctx* ctx, const void* A, int64_t lda, const void* B,
                                       int64_t ldb, const void* const* peers, int64_t ldp, int32_t dest,
                                       const void* residual, int64_t ldr, const void* gamma, float eps,
                                       void* h_out, int64_t ldh, void* y_out, int64_t ldy,
                                       void* partial, int64_t ldc, const entwine_config* cfg,
                                       void* stream);

/* Producer alone (flags still published): partial = bf16(A B).  Used for
 * the uncontended GEMM time of the overlap-efficiency metric (Appendix C). */
entwine_status entwine_gemm_only(entwine_ctx* ctx, const void* A, int64_t lda, const void* B,
                                 int64_t ldb, void* partial, int64_t ldc,
                                 const entwine_config* cfg, void* stream);

/* Reducer alone on an existing partial, every flag published first (the
 * isolated-communication measurement of Appendix A). */
entwine_status entwine_reduce_only(entwine_ctx* ctx, const void* partial, int64_t ldc,
                                   const void* const* peers, int64_t ldp, int32_t dest, void* out,
                                   int64_t ldo, const entwine_config* cfg, void* stream);

/* Per-workgroup timeline of the `back`-th most recent single-launch call
 * made with record_timing (the computation window and communication tail of
 * Section 5.3's figures, per CU): 4 device wall-clock stamps per workgroup
 * {start, producer role end (= start if it had no producer work), first
 * reduction task ready after its waits (0 if it reduced none, and always 0
 * with the layer epilogue), end}, in workgroup order into `stamps`
 * (host, `capacity` entries, at least 4 x nwgs).  nwgs: workgroups of the
 * launch; nproducers: the first nproducers are producers; ticks_per_us: the
 * stamps' clock.  With stamps == NULL only the counts are returned.
 * ENTWINE_EUNSUPPORTED for a call without stamps (two-stream forms, or more
 * than 1024 workgroups).  Blocks until the call completes. */
entwine_status entwine_last_stamps(entwine_ctx* ctx, int32_t back, uint64_t* stamps, int32_t capacity,
                                   int32_t* nwgs, int32_t* nproducers, double* ticks_per_us);

/* Engine clock of the producer role during the `back`-th most recent
 * single-launch call made with record_timing: the engine cycles the producer
 * workgroups counted (s_memtime) over the wall-clock time they spanned,
 * summed over those workgroups, in GHz (host double written to *ghz; 0 if no
 * workgroup produced).  The MFMA peak scales with this clock, which sits
 * below the 2.4 GHz maximum under sustained matrix load and depends on the
 * operand data (Section 5's throughput figures are at whatever clock the
 * device held).  ENTWINE_EUNSUPPORTED for a call without stamps (as for
 * entwine_last_stamps).  Blocks until the call completes. */
entwine_status entwine_last_clock(entwine_ctx* ctx, int32_t back, double* ghz);

/* Waits for the context's queued work, then reports the device status word:
 * returns ENTWINE_ETIMEOUT (with the tile and the flag source, -1 = local,
 * q = peer q) if any reducer wait expired since the previous query, else
 * ENTWINE_OK.  Clears the word.  Any pointer may be NULL. */
entwine_status entwine_query_status(entwine_ctx* ctx, int32_t* code, int32_t* tile, int32_t* src);

/* Event timings of the `back`-th most recent call made with record_timing
 * (0 = latest; at most 255 back): producer kernel time, reducer time from
 * the common start, and end-to-end time (start to the later of the two), in
 * milliseconds.  A value is -1 where the call had no such kernel.  Blocks
 * until those events complete. */
entwine_status entwine_last_timing(entwine_ctx* ctx, int32_t back, float* gemm_ms,
                                   float* reduce_ms, float* e2e_ms);

/* Host-only argument check, the same one every enqueueing call runs. */
entwine_status entwine_validate(int64_t M, int64_t N, int64_t K, int32_t P, int32_t dest,
                                const entwine_config* cfg);

/* Host-only export of the traversal (Equation 1 and the comparison orders)
 * for a BM x BN block grid and a within-partition walk group_m (as in
 * entwine_config, but 0 = N-major here).  blocks: (M/BM)(N/BN) x 4 int32,
 * per logical position p: (d, l, block row, block col).  tiles:
 * (M/128)(N/128) x 2 int32, per global tile in row-major tile order:
 * (partition d, tile number t inside d in producer order).  Either may be
 * NULL. */
entwine_status entwine_tile_schedule(int32_t order, int64_t M, int64_t N, int32_t P, int32_t BM,
                                     int32_t BN, int32_t group_m, int32_t* blocks, int32_t* tiles);

/* Host-only export of the consumer assignment (Section 3.1, "Matching task
 * order"): the partition and tile numbers processed, in order, by reducer
 * workgroup j of x.  dest as in entwine_gemm_rs.  Writes *count tiles to
 * tasks (capacity cap) and the partition to *part. */
entwine_status entwine_consumer_tasks(int32_t dest, int32_t P, int32_t Q, int32_t x, int32_t j,
                                      int32_t* part, int32_t* tasks, int32_t cap, int32_t* count);

const char* entwine_status_string(entwine_status s);
const char* entwine_last_error(const entwine_ctx* ctx);
int32_t entwine_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ENTWINE_H */
