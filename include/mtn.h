/*
 * mtn.h -- C ABI of the windowed-KV frame-attention library (libmtn).
 *
 * The library serves the per-frame attention step of real-time interaction
 * sessions as described by Metronome (arXiv 2607.02640): every session keeps
 * its first S tokens pinned (the attention sinks) plus a sliding window of its
 * last W tokens inside one shared, paged KV pool, and each frame appends a
 * chunk of tokens (chunk prefill, causal inside the chunk and over the
 * retained cache) followed by single-token decode steps.
 *
 *   - Retention and masking: §4.1 and App. A ("Window half", "Sink half").  A
 *     query at absolute position t sees keys k <= t with k < S or k in the W
 *     positions ending at t.
 *   - Positions are absolute and never rebased (§4.1): eviction drops old
 *     keys from memory but never renumbers the ones that stay.
 *   - Frame structure: §2, "The task model" (prefill the chunk, then decode up
 *     to tau tokens), batched over all due sessions (continuous batching).
 *   - Pool: App. A pins ceil(S / block) blocks per session and counts them in
 *     the admission cap; §3 shows that an exhausted pool stalls every session
 *     silently.  Here exhaustion is a loud, atomic error code instead.
 *
 * Conventions for every call:
 *   - Return value: MTN_OK (0) or a negative mtn_status.  On error nothing
 *     changes (host state, device state, out-parameters) unless stated.
 *   - Pointers documented as "device" are HIP device pointers owned by the
 *     caller; "host" pointers are read during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     device work is asynchronous on it; device faults surface at the next
 *     synchronisation.  All calls that belong to one plan must use the same
 *     stream (else MTN_ERR_INVALID_ARG).  A plan may use another stream than
 *     the previous plan: mtn_plan_begin then makes the new stream wait for
 *     everything issued on the previous plan's stream, because plans reuse
 *     the library's device metadata and workspace.  A pool is driven from one
 *     host thread at a time.
 *   - Layouts are row-major with the last index fastest.  The activation
 *     buffers (q, k, v, out of every call and of mtn_frame_batch) must be
 *     16-byte aligned (else MTN_ERR_INVALID_ARG): the kernels move them in
 *     16-byte vectors.
 *   - Element types: MTN_F32 is IEEE binary32, MTN_BF16 is bfloat16.  The KV
 *     cache and q/k/v/out share one element type (kv_dtype == io_dtype),
 *     except for the FP8 cache: kv_dtype MTN_FP8_E4M3 stores every (token,
 *     kv head) row of the rotated key and of the value as OCP E4M3 codes
 *     (bias 7, max 448, round to nearest even) with its own power-of-two
 *     scale 2^e, e the smallest integer with max|row| <= 448 * 2^e (clamped
 *     to [-126, 127], 0 for an all-zero row); its q/k/v/out are bf16
 *     (io_dtype MTN_BF16) and it needs head_dim 128.  Per-token KV
 *     reduction composes with the window bound (Metronome §4.1, closing
 *     remark; §6).  Accumulation is fp32; bf16 results are rounded to
 *     nearest-even.
 */
#ifndef MTN_H
#define MTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t mtn_status;

#define MTN_OK                   0
#define MTN_ERR_INVALID_ARG     (-1)  /* malformed argument or config          */
#define MTN_ERR_BAD_SESSION     (-2)  /* session id not open / out of range    */
#define MTN_ERR_CHUNK_TOO_LARGE (-3)  /* n_tok > max_chunk                     */
#define MTN_ERR_NO_SESSION_SLOT (-4)  /* max_sessions sessions already open    */
#define MTN_ERR_POOL_EXHAUSTED  (-5)  /* windowed: reservation at open fails;
                                         unbounded: a plan needs more blocks   */
#define MTN_ERR_SESSION_FULL    (-6)  /* unbounded: session would pass max_len */
#define MTN_ERR_DEVICE          (-7)  /* a HIP call failed; see last_error     */
#define MTN_ERR_BAD_STATE       (-8)  /* call out of order (plan open/missing,
                                         layer not appended, ...)              */
#define MTN_ERR_UNSUPPORTED     (-9)  /* shape/dtype with no compiled kernel   */
#define MTN_ERR_HOST_MEMORY     (-10) /* a host allocation failed (no C++
                                         exception ever leaves the library)    */

enum { MTN_F32 = 0, MTN_BF16 = 1, MTN_FP8_E4M3 = 2 };

/* window value selecting the unbounded (vanilla) policy: no window, no
 * eviction, sinks ignored, linear block table up to max_len tokens.          */
#define MTN_WINDOW_UNBOUNDED (-1)

/* flags */
#define MTN_POOL_HOST_ONLY 1u /* no device work at all: planning, block tables
                                 and counters only (kv_dev may be NULL); every
                                 append/attend call returns MTN_ERR_BAD_STATE,
                                 plans commit without per-layer appends, and
                                 mtn_frame_step plans without launching        */

typedef struct mtn_pool mtn_pool; /* opaque; owned by the library */

typedef struct {
    int32_t  n_layers;      /* >= 1                                            */
    int32_t  n_q_heads;     /* Hq >= 1                                         */
    int32_t  n_kv_heads;    /* Hkv >= 1, Hq % Hkv == 0; G = Hq / Hkv <= 8      */
    int32_t  head_dim;      /* D: 64 or 128                                    */
    int32_t  block_size;    /* tokens per KV block: must be 16                 */
    int32_t  n_sink;        /* S >= 0 pinned tokens (ignored when unbounded)   */
    int32_t  window;        /* W >= 1, or MTN_WINDOW_UNBOUNDED                 */
    int32_t  max_chunk;     /* C_max >= 1: max tokens per session per plan     */
    int32_t  max_sessions;  /* >= 1 concurrently open sessions                 */
    int32_t  max_len;       /* unbounded only: per-session token cap (>= 1)    */
    int64_t  n_blocks;      /* pool capacity in blocks (>= 1)                  */
    int32_t  kv_dtype;      /* MTN_F32 | MTN_BF16 | MTN_FP8_E4M3               */
    int32_t  io_dtype;      /* kv_dtype, or MTN_BF16 for an MTN_FP8_E4M3 cache */
    double   rope_theta;    /* RoPE base (> 1)                                 */
    float    softmax_scale; /* 0 selects 1/sqrt(head_dim)                      */
    uint32_t flags;         /* MTN_POOL_* flags                                */
} mtn_pool_config;

/*
 * Pool memory.  The caller allocates the KV pool in device memory (e.g. a
 * torch tensor) and keeps it alive until mtn_pool_destroy.  Layout, per layer
 * l, physical block b, KV head h (16 tokens per block, element size e):
 *
 *   K tile   [16][D]  at ((l * n_blocks + b) * Hkv + h) * 2 * 16 * D * e
 *   V^T tile [D][16]  immediately after the K tile
 *
 * K rows hold RoPE-rotated keys; the V tile is stored transposed (dimension-
 * major) so that consecutive tokens of one dimension are adjacent.
 *
 * MTN_FP8_E4M3 (D = 128): each (l, b, h) region is 4224 bytes at
 * ((l * n_blocks + b) * Hkv + h) * 4224 and holds
 *   K codes  [16][128]                       bytes [0, 2048)
 *   V codes  in key quads: byte ((key / 4) * 128 + d) * 4 + key % 4,
 *                                            bytes [2048, 4096)
 *   K exponents e + 127, one byte per key    bytes [4096, 4112)
 *   V exponents e + 127                      bytes [4112, 4128)
 * and 96 bytes of padding; a stored value is code * 2^e.
 */
mtn_status mtn_pool_required_bytes(const mtn_pool_config *cfg, size_t *kv_bytes);

/* One shared, paged KV pool for every session (§4.1: the windowed cache sits
 * in the engine's paged pool; App. A: pinned sink blocks count against its
 * capacity).  Validates cfg, allocates the library's host state and its
 * device metadata and workspace (hipMalloc on the current device; the decode
 * split partials take max_sessions * Hq * 64 * (D + 2) floats), and takes
 * kv_dev (device, caller-owned, >= required bytes, 256-byte aligned) as the
 * pool.  The pool contents are not initialised.  *out receives the handle.
 * Errors: MTN_ERR_INVALID_ARG / MTN_ERR_UNSUPPORTED for cfg, MTN_ERR_DEVICE
 * for a failed HIP allocation, MTN_ERR_HOST_MEMORY; nothing is kept.        */
mtn_status mtn_pool_create(const mtn_pool_config *cfg, void *kv_dev, size_t kv_bytes,
                           void *stream, mtn_pool **out);

/* Frees the library's host and device state (not kv_dev).  Synchronises the
 * device first.  NULL is accepted.                                            */
void mtn_pool_destroy(mtn_pool *pool);

/* Open a session: lowest free session id.  Windowed pools reserve the
 * session's whole bounded footprint, ceil(S/16) sink blocks plus R/16 ring
 * blocks with R = roundup(W + max_chunk - 1, 16), and fail with
 * MTN_ERR_POOL_EXHAUSTED when the reservations would exceed n_blocks (App. A:
 * the admission cap counts the pinned blocks).  Unbounded pools reserve
 * nothing.  Blocks are assigned lazily, lowest free id first.                 */
mtn_status mtn_session_open(mtn_pool *pool, int32_t *sid_out);

/* Close a session: its blocks and reservation return to the pool, its id
 * becomes free.  MTN_ERR_BAD_STATE while a plan is open.                      */
mtn_status mtn_session_close(mtn_pool *pool, int32_t sid);

/*
 * Plans.  Positions advance once per token, not per layer, so per-layer calls
 * act on one open plan:
 *
 *   mtn_plan_begin -> for every layer: mtn_frame_append_kv, then optionally an
 *   attend call -> mtn_plan_commit
 *
 * mtn_plan_begin validates everything first (ids open and unique, 1 <= n_tok
 * <= max_chunk, unbounded max_len and pool capacity), then assigns blocks for
 * the n_tok[i] new positions L_i .. L_i + n_tok[i] - 1 of session sids[i] and
 * uploads the plan (device metadata, RoPE angles) on `stream`.  Planned tokens
 * are packed in plan order: sequence i owns rows off_i .. off_i + n_tok[i] - 1
 * with off_i = n_tok[0] + ... + n_tok[i-1].
 * Slot map: p < S goes to sink block p / 16, offset p % 16; p >= S goes to ring
 * slot (p - S) mod R (unbounded: slot p), i.e. ring block slot / 16, offset
 * slot % 16.  A ring slot is reused only by a position that is R >= W +
 * max_chunk - 1 tokens later, so no key any planned query can see is
 * overwritten (§4.1 per-query window under chunk prefill).
 */
mtn_status mtn_plan_begin(mtn_pool *pool, int32_t n_seq, const int32_t *sids /*host*/,
                          const int32_t *n_tok /*host*/, void *stream);

/* Advance every planned session by its n_tok.  MTN_ERR_BAD_STATE unless every
 * layer was appended (host-only pools excepted).  Positions that leave the window are evicted logically
 * (their slots become reusable); nothing is moved.                            */
mtn_status mtn_plan_commit(mtn_pool *pool);

/* Abandon the open plan instead of committing it, e.g. after a per-layer call
 * failed (failing cleanly instead of stalling every session, §3; or crashing
 * them, App. B).  Every block the plan assigned returns to the pool: block
 * tables, the free list (and so every later lowest-free assignment) and the
 * counters are exactly as before mtn_plan_begin; lengths are unchanged.
 * Device work already issued for the plan is not cancelled; it wrote only
 * slots of positions at or past each session's length, which no later query
 * can see before a later plan has written them again.  MTN_ERR_BAD_STATE
 * when no plan is open.  mtn_frame_step calls it on any error inside a plan. */
mtn_status mtn_plan_abort(mtn_pool *pool);

/*
 * Fused RoPE + append + evict for one layer of the open plan (§4.1: keys keep
 * the absolute position they were appended at; App. A: positions behind the
 * window are not retained, sink blocks stay).
 * k, v: device, [T][Hkv][D] in kv_dtype, T = total planned tokens, packed in
 * plan order.  Each key row is rotated (rotate-half RoPE at its absolute
 * position, angle computed in fp64) and written with its value into the
 * token's slot of layer `layer`, overwriting whatever position left the window
 * there (eviction is slot reuse).  Errors: MTN_ERR_BAD_STATE (no open plan,
 * host-only pool), MTN_ERR_INVALID_ARG (layer, null pointer, stream other
 * than the plan's), MTN_ERR_DEVICE (launch).
 */
mtn_status mtn_frame_append_kv(mtn_pool *pool, int32_t layer, const void *k, const void *v,
                               void *stream);

/*
 * Chunk-prefill attention for one layer of the open plan (after its append):
 * the frame's chunk attends causally inside itself and to the retained cache
 * (§2, the task model; §4.1 and App. A for the per-query mask).
 * q, out: device, [T][Hq][D], packed like k/v.  Each planned query row at
 * position t is rotated at t and attends to sinks [0, min(S, t+1)) and window
 * [max(S, t-W+1), t] of its own session (all earlier chunk tokens included).
 * lse: device [T][Hq] fp32 natural-log sum-exp of the scaled scores, or NULL.
 * bf16 pools run the MFMA kernel, fp32 pools the fp32 vector kernel.
 */
mtn_status mtn_attend_chunk_prefill(mtn_pool *pool, int32_t layer, const void *q, void *out,
                                    float *lse, void *stream);

/*
 * GQA decode attention for one layer of the open plan, whose every sequence
 * has n_tok == 1.  q, out: device, [n_seq][Hq][D]; lse: device [n_seq][Hq] or
 * NULL.  The G query heads sharing a KV head read its sinks ∪ window once;
 * n_split > 1 splits the keys into segments merged by log-sum-exp, sinks in
 * segment 0 only (App. A segmented decode).  n_split = 0 picks a split from
 * the batch size; 1 <= n_split <= 64 forces it (the workspace holds 64
 * segments of every query; mtn_pool_last_split reports the split used).
 */
mtn_status mtn_attend_decode(mtn_pool *pool, int32_t layer, const void *q, void *out,
                             float *lse, int32_t n_split, void *stream);

/*
 * mtn_attend_decode for callers that cannot allocate device memory (code
 * under HIP graph capture, allocation-free serving loops, harnesses that
 * forbid hipMalloc): same arguments, layouts and results, but the split
 * partials live in a static device array of the library (4 Mi floats = 16
 * MiB, one per GPU, held until the process ends) instead of the pool's
 * workspace, and the call allocates nothing and records no timing events.
 * A forced split needs n_seq * Hq * n_split * (D + 2) <= 4 Mi floats, else
 * MTN_ERR_INVALID_ARG; n_split = 0 picks the automatic split, reduced to what
 * the array holds.  Every call on one GPU shares the array: calls that
 * overlap on one GPU (two streams, two pools) race and must be ordered by
 * the caller.
 */
mtn_status mtn_attend_decode_noalloc(mtn_pool *pool, int32_t layer, const void *q, void *out,
                                     float *lse, int32_t n_split, void *stream);

/*
 * mtn_frame_append_kv followed by mtn_attend_decode for one layer of an open
 * plan whose every sequence has n_tok == 1, in one launch: each planned token
 * is the newest key of its own query, so the workgroup that attends to the
 * end of that query's window takes the new key and value from k / v
 * (rotated and rounded exactly as the stored copy) and writes the stored
 * copy for later calls.  Same arguments and layouts as the two calls; the
 * layer must not have been appended yet in this plan (MTN_ERR_BAD_STATE).
 * mtn_frame_step uses this form for its decode rounds.
 */
mtn_status mtn_attend_decode_append(mtn_pool *pool, int32_t layer, const void *k, const void *v,
                                    const void *q, void *out, float *lse, int32_t n_split,
                                    void *stream);

/*
 * One whole frame for a batch of sessions (§2 task model): plan the chunk,
 * then for each layer append + chunk-prefill attend, commit; then for each
 * decode round j (only sessions with n_decode[i] > j) plan one token, for each
 * layer append + decode attend (one launch, as mtn_attend_decode_append),
 * commit.  Chunks of one token everywhere use the decode kernel the same way.
 * With the fp8 pool, when every sequence's chunk rows fit one prefill row
 * pass (and the launch is small enough), the chunk append runs inside the
 * prefill's launch; the pool holds the same bytes either way.
 * Every host check (sessions, sizes, and block capacity for the whole frame)
 * runs before the first plan.  An error inside a plan (a failed launch)
 * abandons that plan as mtn_plan_abort does; plans of the frame that already
 * committed stay committed (each session's length tells how far it got), and
 * output rows of unfinished plans are undefined.  On a host-only pool the
 * frame is planned and committed without device work (buffers may be NULL).
 */
typedef struct {
    int32_t        n_seq;
    const int32_t *sids;       /* host [n_seq]                                */
    const int32_t *chunk_len;  /* host [n_seq], 1 <= chunk_len <= max_chunk   */
    const int32_t *n_decode;   /* host [n_seq], >= 0                          */
    /* device [n_layers][sum(chunk_len)][H][D], rows packed in batch order    */
    const void *q_chunk, *k_chunk, *v_chunk;
    void       *out_chunk;     /* [n_layers][sum(chunk_len)][Hq][D]           */
    float      *lse_chunk;     /* [n_layers][sum(chunk_len)][Hq] or NULL      */
    /* device [max(n_decode)][n_layers][n_seq][H][D]; entry (j, l, i) is read
     * (written) only when n_decode[i] > j                                    */
    const void *q_dec, *k_dec, *v_dec;
    void       *out_dec;       /* [max(n_decode)][n_layers][n_seq][Hq][D]     */
    float      *lse_dec;       /* [max(n_decode)][n_layers][n_seq][Hq] or NULL */
    int32_t     n_split;       /* decode split, 0 = automatic                 */
} mtn_frame_batch;

mtn_status mtn_frame_step(mtn_pool *pool, const mtn_frame_batch *batch, void *stream);

/* ---- observability and test hooks ------------------------------------- */

typedef struct {
    int64_t capacity;       /* n_blocks                                        */
    int64_t assigned;       /* blocks currently holding session data           */
    int64_t reserved;       /* windowed: sum of open reservations; unbounded:
                               equal to assigned                               */
    int32_t open_sessions;
    int32_t blocks_per_session; /* row length of the block table              */
    int32_t ring_tokens;    /* R                                               */
    int32_t sink_blocks;    /* ceil(S / 16) (0 when unbounded)                 */
} mtn_pool_stats_t;

mtn_status mtn_pool_stats(const mtn_pool *pool, mtn_pool_stats_t *out);

/* Length (tokens appended so far, committed) and assigned block count. */
mtn_status mtn_session_info(const mtn_pool *pool, int32_t sid, int64_t *len,
                            int32_t *n_assigned);

/* Copy the session's block-table row (-1 = unassigned) into host out[cap];
 * *n_out receives the row length.  MTN_ERR_INVALID_ARG if cap is too small. */
mtn_status mtn_session_block_table(const mtn_pool *pool, int32_t sid, int32_t *out,
                                   int32_t cap, int32_t *n_out);

/* For the open plan: host arrays of length >= T receive, per planned token,
 * its absolute position, physical block and offset (any pointer may be NULL);
 * evicted_lo/hi (length >= n_seq, may be NULL) receive each sequence's
 * half-open range of positions that leave the window at commit.  *n_tok_out
 * receives T.                                                                */
mtn_status mtn_plan_info(const mtn_pool *pool, int64_t *pos, int32_t *block, int32_t *offset,
                         int32_t cap, int64_t *evicted_lo, int64_t *evicted_hi,
                         int32_t *n_tok_out);

/* Debug: write NaN into every slot that no query may read: all unassigned
 * blocks, sink-block slots at or past S, and ring slots of positions outside
 * each open session's retained set.  Attention results must not change.       */
mtn_status mtn_debug_poison_dead(mtn_pool *pool, void *stream);

/* Tuning: query rows per chunk-prefill pass (rows are token x G + group head;
 * each pass of each kv head is one workgroup that reads the keys its rows can
 * see).  0 (the default) chooses per plan: 256, or 128 when the plan's 256-row
 * passes would occupy at most half the GPU's compute units; 128 or 256 fix it.
 * Takes effect at the next mtn_plan_begin.  Results are the same either way
 * up to fp32 summation order.  Other values: MTN_ERR_INVALID_ARG.            */
mtn_status mtn_pool_set_prefill_pass_rows(mtn_pool *pool, int32_t rows);

/* Test / tuning: the decode kernel.  0 (default) chooses by shape; 1 forces
 * the vector kernel (fp32 and bf16 pools); 2 forces the matrix-core kernel
 * (bf16 pools with head_dim 128; FP8 pools always use it).  Takes effect at
 * the next launch; results agree up to fp32 summation order.
 * MTN_ERR_UNSUPPORTED where the kernel does not exist for the pool,
 * MTN_ERR_BAD_STATE while a plan is open.                                    */
mtn_status mtn_pool_set_decode_kernel(mtn_pool *pool, int32_t kind);

/* Key segments (split) of the most recent decode launch of this pool.        */
mtn_status mtn_pool_last_split(const mtn_pool *pool, int32_t *n_split);

/* Test hook: the launch point with index launch_index (0 = the next one)
 * among this pool's later append / prefill / decode launch points fails with
 * MTN_ERR_DEVICE before launching; -1 disarms.  Host-only pools pass through
 * the same points inside mtn_frame_step, so error paths can be exercised on a
 * host without a GPU.                                                        */
mtn_status mtn_debug_inject_failure(mtn_pool *pool, int64_t launch_index);

/* Per-kernel device timing.  When enabled, the library records HIP events
 * around each launch it makes and accumulates per-kernel-class totals;
 * mtn_pool_kernel_times synchronises those events and returns, for classes
 * 0 append, 1 prefill, 2 decode, 3 merge, the launch count and the summed
 * milliseconds (arrays of length >= 4), then resets the totals.               */
mtn_status mtn_pool_set_timing(mtn_pool *pool, int32_t enable);
mtn_status mtn_pool_kernel_times(mtn_pool *pool, int64_t *launches, double *ms);

/* Plain device copy (dst = src, `bytes` a multiple of 16, both 16-byte
 * aligned): the bandwidth reference for the HBM roofline and the scale of the
 * profiler's byte counters.                                                   */
mtn_status mtn_hbm_copy(const void *src, void *dst, size_t bytes, void *stream);

/* Device read of `bytes` (a multiple of 8192, src 16-byte aligned) through the
 * same non-temporal LDS DMA the decode streams its blocks with: 8 KiB chunks
 * interleaved over the waves, two in flight per wave, nothing computed or
 * written.  The achievable read bandwidth of that mechanism, the ceiling
 * beside the nominal HBM peak for the decode.                               */
mtn_status mtn_hbm_read(const void *src, size_t bytes, void *stream);

/* ---- deadline-aware admission (host only) ------------------------------ */

/*
 * An AIMD admission controller on the measured per-frame latency (§4.2: the
 * schedulable concurrency depends on model, window, hardware and arrivals, so
 * it is discovered from feedback instead of set by hand; arrivals beyond the
 * cap get a clean rejection).  The caller offers each arriving session, opens
 * a pool session only when it is admitted, releases it when the session ends,
 * and reports every tick's latency (e.g. the time of one mtn_frame_step over
 * all admitted sessions).  Per observed tick:
 *   - during `hold` observations after a cut, nothing changes (the cut must
 *     reach the signal first);
 *   - latency >= target_ms: cap = max(min_cap, min(cap, floor(backoff *
 *     admitted))) -- a multiplicative cut relative to the load that produced
 *     the latency; admitted sessions are never evicted;
 *   - otherwise, if since the previous observation an offer was rejected or
 *     the admitted count reached the cap: cap = min(max_cap, cap + increase).
 * An offer is admitted iff admitted < cap.  All arithmetic is IEEE double and
 * int32; the controller is deterministic given the call sequence.
 * A controller is used from one host thread.
 */
typedef struct mtn_admission mtn_admission; /* opaque; owned by the library */

typedef struct {
    double  target_ms;    /* latency target, > 0 (e.g. 0.3 x the frame budget)   */
    double  backoff;      /* multiplicative factor, 0 < backoff < 1               */
    int32_t increase;     /* additive step per observation, >= 1                  */
    int32_t initial_cap;  /* min_cap <= initial_cap <= max_cap                    */
    int32_t min_cap;      /* >= 1                                                 */
    int32_t max_cap;
    int32_t hold_ticks;   /* observations without a decision after a cut, >= 0   */
} mtn_admission_config;

typedef struct {
    int32_t cap;          /* current admission cap                                */
    int32_t admitted;     /* admitted and not yet released                        */
    int32_t hold;         /* observations left before the next decision           */
    int64_t offered, rejected, ticks, decreases, increases;
} mtn_admission_state;

/* MTN_ERR_INVALID_ARG for a config outside the ranges above. */
mtn_status mtn_admission_create(const mtn_admission_config *cfg, mtn_admission **out);
void       mtn_admission_destroy(mtn_admission *a);          /* NULL accepted   */
/* One arriving session: *admitted = 1 (admitted, counted) or 0 (rejected).    */
mtn_status mtn_admission_offer(mtn_admission *a, int32_t *admitted);
/* An admitted session ended.  MTN_ERR_BAD_STATE when none is admitted.        */
mtn_status mtn_admission_release(mtn_admission *a);
/* One tick's latency in ms (finite, >= 0): the AIMD update above.             */
mtn_status mtn_admission_observe(mtn_admission *a, double tick_ms);
mtn_status mtn_admission_get(const mtn_admission *a, mtn_admission_state *out);

const char *mtn_status_string(mtn_status s);
const char *mtn_pool_last_error(const mtn_pool *pool);

#ifdef __cplusplus
}
#endif
#endif /* MTN_H */
