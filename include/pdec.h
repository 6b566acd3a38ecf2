/*
 * pdec — event-parallel decode attention for AMD MI355X (gfx950).
 *
 * One decode step of the event-factorized parallel decoding of PadCaptioner
 * (arXiv 2607.02963, §3.4, Eq. 3): E event caption streams each issue one
 * query token at once.  Every query attends to
 *   (1) the shared prefix of its video: the audio-visual tokens, the
 *       instruction and the latent global-plan tokens G^1..G^K (§3.1, §3.3),
 *       all fully visible, and
 *   (2) the rows of its own stream's cache: its anchor and the local tokens it
 *       generated so far, the newest row being the current token;
 * and never the rows of another stream (the §3.4 mask, Fig. 3).  Streams stop
 * independently at EOS (§3.4, last paragraph); a stopped stream has no query.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are dense, row-major, in device memory, 16-byte aligned, of the
 *    element type named by pdec_dims.dtype (float32, or bfloat16 stored as
 *    16-bit words).  Integer arrays (lengths, offsets, flags) are int32 in
 *    device memory, 4-byte aligned; so is lse.
 *  - q, out    [num_events, H_q, D]        one row per stream
 *    lse       [num_events, H_q]  float32  natural-log log-sum-exp of the
 *                                          scaled scores of that row
 *    k/v_prefix [prefix rows, H_kv, D]     token-major, as a KV cache stores it
 *    k/v_event  [num_events, event_cap, H_kv, D]  one cache per stream
 *  - Query head h reads key/value head h / (H_q / H_kv).
 *  - event_lens[e] = n_e, the number of visible rows of stream e's cache,
 *    INCLUDING the current token (append first, then attend).  n_e == 0 means
 *    the stream has ended: its out row is written as 0 and its lse as -inf.
 *  - Scores are softmax_scale * <q, k>; softmax_scale <= 0 selects 1/sqrt(D).
 *  - Accumulation is float32 whatever the input type; out is rounded to the
 *    input type (round to nearest even for bfloat16).
 *  - The caller owns every buffer.  No entry point allocates or frees device
 *    memory; the step calls use only the caller's workspace.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL is the null
 *    stream) and makes no implicit synchronisation.  Host-checkable argument
 *    errors are reported before anything is enqueued.  Lengths held in device
 *    memory are a caller contract (0 <= n_e <= event_cap, 0 <= prefix length
 *    <= max_prefix_len, non-decreasing offsets); they are not checked.
 *  - Calls sharing one workspace must not overlap in time.
 *  - Debug mode: with the environment variable PDEC_DEBUG=1 (read once, when
 *    the library is first used), the step calls copy the device lengths to the
 *    host (synchronising `stream`), check them with pdec_check_lengths, and
 *    return PDEC_ERR_BAD_LENGTHS before launching anything if they break the
 *    contract.  Off by default: a step then never synchronises.
 */
#ifndef PDEC_H
#define PDEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PDEC_OK = 0,
    PDEC_ERR_INVALID_ARG = -1, /* null / misaligned pointer, inconsistent sizes          */
    PDEC_ERR_UNSUPPORTED = -2, /* a size or type this build has no kernel for (D, dtype) */
    PDEC_ERR_WORKSPACE = -3,   /* workspace smaller than pdec_workspace_size()          */
    PDEC_ERR_HIP = -4,         /* a HIP runtime call or kernel launch failed             */
    PDEC_ERR_BAD_LENGTHS = -5, /* a length held in device memory breaks the contract     */
                               /* (only detected with PDEC_DEBUG=1, see below)           */
    PDEC_ERR_SCRATCH = -6      /* the step needs more scratch than the library's static  */
                               /* buffer holds (pdec_attn_step_noalloc only)             */
} pdec_status;

typedef enum { PDEC_DTYPE_F32 = 0, PDEC_DTYPE_BF16 = 1 } pdec_dtype;

/* Sizes of one call.  All fields are host values. */
typedef struct pdec_dims {
    int32_t num_events;           /* rows of q/out/lse: E of one video, or the total over videos */
    int32_t num_q_heads;          /* H_q, a multiple of num_kv_heads                             */
    int32_t num_kv_heads;         /* H_kv                                                        */
    int32_t head_dim;             /* D: 64 or 128                                                */
    int32_t event_cap;            /* rows per stream cache, >= 1                                 */
    int32_t max_prefix_len;       /* upper bound on any video's prefix length, >= 0              */
    int32_t max_events_per_video; /* upper bound on streams in one video (<= 2048); 0 means      */
                                  /* min(num_events, 2048)                                       */
    int32_t dtype;                /* pdec_dtype of q, k, v and out                               */
    float softmax_scale;          /* <= 0 selects 1/sqrt(head_dim)                               */
    int64_t prefix_tokens;        /* prefix rows over the whole batch (sizing hint for the work  */
                                  /* split); 0 means num_videos * max_prefix_len                 */
    int32_t plan_mask;            /* 0: every stream sees the whole prefix, plan tokens included */
                                  /* (§3.4, the full design).  1: the "self G-token only" mask   */
                                  /* of Table 8: of the plan segment a stream sees only its own  */
                                  /* global tokens                                               */
    int32_t plan_tokens_per_stream; /* T, used when plan_mask = 1: the plan segment of a video  */
                                  /* with E streams is its last E*T prefix tokens, stream f's    */
                                  /* global tokens being the f-th run of T; E counts every      */
                                  /* stream slot of the video, ended ones included.  The mask   */
                                  /* is meant for E*T <= L; beyond that the runs keep their     */
                                  /* places counted from L - E*T and the parts before prefix    */
                                  /* key 0 do not exist.  0 means no plan segment.  Must be >= 0 */
    int32_t queries_per_stream;   /* Q; 0 or 1: one query per stream, the decode step.  Q > 1:   */
                                  /* whole branches at once (the prefill / training form of     */
                                  /* §3.4's mask, Fig. 3): q and out are [num_events, Q, H_q, D], */
                                  /* lse [num_events, Q, H_q], and query j of stream e sees the   */
                                  /* prefix and its own rows 0 .. min(j, n_e - 1), never another  */
                                  /* stream's; n_e == 0 gives rows of 0 / -inf.  Q > 1 needs      */
                                  /* bfloat16 and plan_mask == 0 (else PDEC_ERR_UNSUPPORTED).    */
    int32_t cross_causal;         /* 0: the event-factorized mask.  1: the "causal attention" row */
                                  /* of Table 8 (whole branches only, queries_per_stream > 1):   */
                                  /* the tokens of one step share a position (§3.4), so query j */
                                  /* also sees every other stream's rows t < min(j, n_f).        */
} pdec_dims;

/* Human-readable text of a pdec_status code.  Never NULL. */
const char* pdec_strerror(int status);

/*
 * Bytes of workspace a step call with these dims needs (num_videos = 1 for
 * pdec_attn_step).  The workspace holds the per-chunk partial softmax states
 * (running max and normaliser in float32, and the normalised output in the
 * inputs' element type, per query row) that the split of the prefix across
 * compute units produces.  Returns 0 if the dims
 * are invalid.  Pure host function: touches no device.
 */
size_t pdec_workspace_size(const pdec_dims* dims, int32_t num_videos);

/*
 * One parallel decode step for one video (§3.4, Eq. 3).
 *   q           [E, H_q, D]            current query of every stream
 *   k_prefix, v_prefix [>= L, H_kv, D] shared prefix cache of the video
 *                      (may be NULL when dims->max_prefix_len == 0)
 *   k_event, v_event   [E, event_cap, H_kv, D]
 *   event_lens  [E]  int32, device     n_e per stream (see conventions)
 *   prefix_lens [1]  int32, device     L, 0 <= L <= dims->max_prefix_len
 *   out         [E, H_q, D]            written for every row
 *   lse         [E, H_q] float32, or NULL to skip it
 *   workspace   device, >= pdec_workspace_size(dims, 1) bytes, contents ignored
 * E = dims->num_events.  With dims->queries_per_stream = Q > 1 the call
 * evaluates whole branches: q and out are [E, Q, H_q, D], lse [E, Q, H_q]
 * (see pdec_dims).  Returns a pdec_status.
 */
int pdec_attn_step(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                   const void* k_event, const void* v_event, const int32_t* event_lens,
                   const int32_t* prefix_lens, void* out, float* lse, void* workspace,
                   size_t workspace_bytes, void* stream);

/*
 * pdec_attn_step for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, semantics and kernels as pdec_attn_step, but the partial
 * softmax states live in a scratch buffer the library holds in static device
 * memory: PDEC_NOALLOC_SCRATCH_BYTES (32 MiB) on every GPU the library runs
 * on, kept until the process ends.  The call allocates and frees nothing
 * (no hipMalloc / hipFree, no allocating library routine).  A step whose
 * workspace would exceed the buffer (pdec_workspace_size(dims, 1) >
 * PDEC_NOALLOC_SCRATCH_BYTES) is refused with PDEC_ERR_SCRATCH before
 * anything is enqueued.  The prefix 32768 / 32-stream step needs about 15 MiB.
 * Every call on one GPU shares that GPU's buffer: calls that overlap in time
 * on one GPU (from several streams or threads) race on it and must be
 * serialised by the caller.  The first call on a device looks up the
 * buffer's address there (a host-side query, no allocation).  Returns a
 * pdec_status.
 */
#define PDEC_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int pdec_attn_step_noalloc(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                           const void* k_event, const void* v_event, const int32_t* event_lens,
                           const int32_t* prefix_lens, void* out, float* lse, void* stream);

/*
 * One parallel decode step over a ragged batch of videos, every (video,
 * stream) pair at once.  Video v owns prefix rows [cu_prefix[v],
 * cu_prefix[v+1]) of the packed k/v_prefix and streams [cu_events[v],
 * cu_events[v+1]) of q/out/lse and of the stream caches.  Streams of one video
 * never see another video's prefix or streams.
 *   cu_prefix, cu_events [num_videos + 1] int32, device, starting at 0;
 *   cu_events[num_videos] == dims->num_events; every per-video prefix length
 *   <= dims->max_prefix_len and stream count <= dims->max_events_per_video.
 *   workspace >= pdec_workspace_size(dims, num_videos) bytes.
 * Other arguments as for pdec_attn_step.  Returns a pdec_status.
 */
int pdec_attn_step_ragged(const pdec_dims* dims, int32_t num_videos, const void* q,
                          const void* k_prefix, const void* v_prefix, const int32_t* cu_prefix,
                          const void* k_event, const void* v_event, const int32_t* event_lens,
                          const int32_t* cu_events, void* out, float* lse, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * A decode step with the cache append fused into it (§3.4: at each step every
 * live stream appends its own new token and attends; a stream that has
 * emitted EOS stops while the others go on).  Equivalent to pdec_kv_append
 * followed by a step call, bit for bit, in one pass over the caches:
 *   - lens_in[e] holds the counts BEFORE this step's append.  For a stream
 *     with live[e] != 0 (every stream when live is NULL) whose cache has
 *     room, lens_in[e] < event_cap, the step attends lens_in[e] + 1 own rows,
 *     the last being k_new[e] / v_new[e], which are also written into cache
 *     row lens_in[e]; a live stream with a full cache attends its
 *     lens_in[e] rows and appends nothing; a stream with live[e] == 0 has
 *     ended (out row 0, lse -inf).
 *   - lens_out[e] receives the counts after the append (lens_in[e] + 1, the
 *     same, or 0 for an ended stream).  lens_out must not be lens_in: no
 *     work-group reads a count another one writes, so a loop swaps the two
 *     arrays between steps.
 *   - k_new, v_new [E, H_kv, D] device, 16-byte aligned, read;
 *     k_event, v_event [E, event_cap, H_kv, D] device, read, and row
 *     lens_in[e] of every appending stream written;  live [E] int32 or NULL.
 *   - One video: num_videos 1, prefix_lens [1] device, cu_prefix and
 *     cu_events NULL.  A batch: cu_prefix and cu_events as for
 *     pdec_attn_step_ragged, prefix_lens ignored.
 *   - q, k_prefix, v_prefix, out, lse, workspace as for pdec_attn_step.
 * dims->queries_per_stream must be 0 or 1 (else PDEC_ERR_UNSUPPORTED).  The
 * 32-row-tile kernels (pdec_set_path(3)) are not used by this call.
 * PDEC_DEBUG=1 checks lens_in.  Asynchronous on `stream`.  Returns a
 * pdec_status.
 */
int pdec_decode_step(const pdec_dims* dims, int32_t num_videos, const void* q, const void* k_prefix,
                     const void* v_prefix, const int32_t* prefix_lens, const int32_t* cu_prefix,
                     const int32_t* cu_events, const void* k_new, const void* v_new, void* k_event, void* v_event,
                     const int32_t* lens_in, int32_t* lens_out, const int32_t* live, void* out, float* lse,
                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * Per-stream cache append before a step (§3.4: each live stream extends its
 * own subchain; App. B.5: the total cache does not grow beyond what
 * sequential decoding would hold).  For every stream e with live[e] != 0
 * (or every stream when live is NULL): row n = event_lens[e] of its caches
 * receives k_new[e] / v_new[e] ([H_kv, D] each) and event_lens[e] becomes
 * n + 1.  For a stream with live[e] == 0, nothing is written and
 * event_lens[e] becomes 0 (the stream has ended).  A live stream whose cache
 * is full (n >= event_cap) is left unchanged.
 *   k_new, v_new [E, H_kv, D];  k_event, v_event [E, event_cap, H_kv, D];
 *   event_lens [E] int32, device, read and written;  live [E] int32 or NULL.
 * E = dims->num_events.  Returns a pdec_status.
 */
int pdec_kv_append(const pdec_dims* dims, const void* k_new, const void* v_new, void* k_event,
                   void* v_event, int32_t* event_lens, const int32_t* live, void* stream);

/*
 * The append fused with the rotary position embedding at the shared decode
 * position (§3.4: the tokens of all streams at one decoding step carry one
 * position index).  For every stream e with live[e] != 0 (or every stream
 * when live is NULL) whose cache has room, n = event_lens[e] < event_cap:
 *   pos = pos_base[v] + n, v the stream's video;
 *   q[e, h] is rotated by R(pos) in place, for every query head;
 *   cache row n of k_event receives R(pos) k_new[e], of v_event v_new[e];
 *   event_lens[e] becomes n + 1.
 * A stream with live[e] == 0 gets event_lens[e] = 0 and nothing else; a live
 * stream with a full cache is left unchanged, its q included.
 * R(pos) turns coordinates (i, i + D/2) of a head by pos * rope_theta^(-2i/D),
 * i < D/2 (the rotate-half form: y_i = x_i cos - x_{i+D/2} sin,
 * y_{i+D/2} = x_{i+D/2} cos + x_i sin).  Angles and products are computed in
 * double and rounded once to the element type (nearest even).
 *   q [E, H_q, D] read and written;  k_new, v_new [E, H_kv, D];
 *   k_event, v_event [E, event_cap, H_kv, D];  event_lens [E] read and written;
 *   live [E] int32 or NULL;  cu_events [num_videos + 1] int32 (streams of
 *   video v are [cu_events[v], cu_events[v+1])) or NULL for one video;
 *   pos_base [num_videos] int32;  all device.  rope_theta > 0, finite.
 * E = dims->num_events.  Returns a pdec_status.
 */
int pdec_rope_kv_append(const pdec_dims* dims, int32_t num_videos, void* q, const void* k_new,
                        const void* v_new, void* k_event, void* v_event, int32_t* event_lens,
                        const int32_t* live, const int32_t* cu_events, const int32_t* pos_base,
                        float rope_theta, void* stream);

/*
 * Kernel-path selection for the shared-prefix pass, for tests and tuning:
 * 0 = automatic (bfloat16 uses the matrix-core kernel, float32 the vector
 * kernel), 1 = always the
 * vector kernel, 2 = matrix-core kernel where the type allows it, 3 = as 2,
 * with the decode step at head_dim 128 and more than 64 query rows per kv
 * head on 32-row tiles (kernel shapes 4 and 5) instead of 16-row ones.
 * Process-wide; returns the previous setting, or PDEC_ERR_INVALID_ARG.
 */
int pdec_set_path(int path);

/*
 * The kernel path (1 = vector, 2 = matrix core) and the prefix chunk length
 * (keys per work item) a step call with these dims would use.  Host-only.
 * Returns a pdec_status.
 */
int pdec_query_plan(const pdec_dims* dims, int32_t num_videos, int32_t* path, int32_t* chunk_keys);

/* The whole work split of a step call, for tests and measurement. */
typedef struct pdec_plan_info {
    int32_t path;          /* 1 = vector kernel, 2 = matrix-core kernel                          */
    int32_t kernel_shape;  /* matrix-core work-group shape: 1 = 64 rows, 2 = 128 rows,          */
                           /* 3 = 256 rows on 16-row tiles; 4 = 256 rows, 5 = 128 rows on      */
                           /* 32-row tiles (pdec_set_path(3) only); 0 on the vector path       */
    int32_t rows_per_item; /* query rows of one kv head that one work item serves               */
    int32_t row_groups;    /* work items per (video, kv head, chunk): ceil(rows / rows_per_item)  */
    int32_t chunk_keys;    /* keys of the virtual key sequence per chunk                         */
    int32_t max_chunks;    /* partial-state slots per row: the chunks, plus slot 0 of the tail   */
                           /* pass when tail_blocks > 0                                          */
    int32_t work_items;    /* work items of the split pass (prefix chunks x row groups x heads) */
    int32_t merge_pass;    /* 1 if partial states are merged after the split pass, else 0 (the  */
                           /* split pass writes out and lse itself)                              */
    int32_t tail_blocks;   /* work-groups of the per-stream tail pass in the split launch (each */
                           /* (stream, kv head) pair's G rows against the stream's own keys, 8  */
                           /* pairs per work-group); 0 when the own keys are chunk units        */
} pdec_plan_info;

/*
 * Fills *info with the plan a step call with these dims would use
 * (num_videos = 1 for pdec_attn_step).  Host-only.  Returns a pdec_status;
 * PDEC_ERR_INVALID_ARG for a NULL info or invalid dims.
 */
int pdec_describe_plan(const pdec_dims* dims, int32_t num_videos, pdec_plan_info* info);

/*
 * Measurement hook.  With n > 0, the i-th step call made after this call
 * brackets its split pass (the kernel that reads the shared prefix and the
 * stream caches) with hipEventRecord(start_events[i % n]) and
 * hipEventRecord(stop_events[i % n]) on the call's stream, so a caller can
 * time that kernel alone without changing the work done.  The events are
 * hipEvent_t handles owned by the caller.  n = 0 (or NULL arrays) turns the
 * hook off.  Process-wide; the hook's state is guarded by a lock, so step
 * calls from several threads each take their own event pair (in call order).
 * Returns a pdec_status.
 */
int pdec_set_split_timer(void* const* start_events, void* const* stop_events, int n);

/*
 * The device-length contract, checked on HOST copies of the length arrays
 * (the check PDEC_DEBUG=1 runs before a step): 0 <= event_lens[e] <=
 * event_cap for every stream; with num_videos == 1, prefix_lens[0] in
 * [0, max_prefix_len]; with num_videos > 1, cu_prefix and cu_events start at
 * 0, never decrease, end at the total prefix rows (when dims->prefix_tokens
 * > 0) and at num_events, and each video's prefix (cu_prefix[v+1] -
 * cu_prefix[v]) is at most max_prefix_len and its stream count at most
 * max_events_per_video (when > 0).  Pass prefix_lens for one video, or
 * cu_prefix and cu_events for a ragged batch.  Returns PDEC_OK,
 * PDEC_ERR_BAD_LENGTHS, or PDEC_ERR_INVALID_ARG for invalid dims or missing
 * arrays.  Host-only; reads num_events + num_videos + 1 values at most.
 */
int pdec_check_lengths(const pdec_dims* dims, int32_t num_videos, const int32_t* event_lens,
                       const int32_t* prefix_lens, const int32_t* cu_prefix, const int32_t* cu_events);

/*
 * Measurement aid (the read ceiling the split pass is compared with): streams
 * a K/V cache pair of the decode step's layout, k and v each [L, H_kv, 128]
 * bfloat16 in device memory (16-byte aligned), once, computing nothing.
 *   mode 0: plain 16-byte loads, each work-group a contiguous slab (the
 *           HBM read ceiling for these bytes in one launch);
 *   mode 1: the decode split pass's memory path: items of (kv head,
 *           keys_per_item keys, a multiple of 64), every 64-key stage of the
 *           head's key and value rows moved into a 3-slot LDS ring (two stages
 *           in flight) by direct-to-LDS loads with a work-group barrier per
 *           stage.
 * sink: device int32, written only when the data hash to a fixed value (so
 * the reads cannot be optimised away).  Asynchronous on `stream`.  Returns
 * PDEC_ERR_INVALID_ARG for null or misaligned pointers, L or H_kv < 1, a mode
 * other than 0 or 1, or (mode 1) keys_per_item not a positive multiple of 64.
 */
/*
 * Measurement aid (why the split kernel's stages take the sum of their
 * matrix and vector work): 256 work-groups of 64 * 4 * waves_per_simd lanes
 * (waves_per_simd 1, 2 or 4 waves on each of a compute unit's four SIMDs),
 * each wave running `iters` iterations of a fixed instruction block:
 *   mode 0: eight independent v_mfma_f32_16x16x32_bf16;
 *   mode 1: thirty-two v_fma_f32 over eight independent registers;
 *   mode 2: both blocks in every wave, one after the other;
 *   mode 3: half the waves of each SIMD the matrix block, half the vector
 *           block (waves_per_simd 2 or 4).
 * Time the launch on `stream` (HIP events): with both kinds of work on a SIMD
 * the time is the sum of the parts when the two do not overlap, their
 * maximum when they do.  sink: a device float, written only in a case that
 * the inputs never reach.  Asynchronous.  Returns PDEC_ERR_INVALID_ARG for a
 * null or misaligned sink, a mode outside 0..3, iters < 1, waves_per_simd
 * not 1, 2 or 4, or mode 3 with one wave per SIMD.
 */
int pdec_issue_probe(int32_t mode, int32_t waves_per_simd, int32_t iters, float* sink, void* stream);

int pdec_read_probe(const void* k, const void* v, int32_t L, int32_t H_kv, int32_t keys_per_item, int32_t mode,
                    int32_t* sink, void* stream);

/*
 * Segment-level similarity grounding at inference (App. "More Implementation
 * Details": grounding by feature similarity).  For the K generated global
 * event tokens of a video and its N audio-visual prefix tokens, both already
 * projected by the caller's two-layer MLP to width d:
 *   score[i, s]   = sum over tokens n of segment s of <g_i, p_n>,
 *   salient[i, s] = 1 if score[i, s] > threshold * max over s' of score[i, s'],
 *                   else 0   (threshold 0.5 or 0.7 in the paper's experiments).
 * Segment s is the contiguous token range [cu_seg[s], cu_seg[s+1]); an empty
 * segment scores 0.  Scores accumulate in float32; each segment adds its
 * per-chunk pieces in a fixed order, so repeated calls agree bit for bit.
 */
typedef struct pdec_ground_dims {
    int32_t num_events;    /* K, 1..64                                              */
    int32_t num_tokens;    /* N >= 1                                                */
    int32_t num_segments;  /* S >= 1                                                */
    int32_t dim;           /* d: 64, 128 or 256                                     */
    int32_t dtype;         /* PDEC_DTYPE_BF16 (the only type with a kernel)         */
} pdec_ground_dims;

/* Workspace bytes for pdec_segment_grounding (0 for invalid dims). Host only. */
size_t pdec_grounding_workspace_size(const pdec_ground_dims* dims);

/*
 *   g [K, d], p [N, d]           device, bf16, rows contiguous, 16-byte aligned;
 *   cu_seg [S + 1] int32         device, non-decreasing from 0 to N (not checked:
 *                                ranges are clamped to [0, N), so a bad table gives
 *                                wrong scores, never a stray access);
 *   scores [K, S] float32, salient [K, S] uint8   device, written;
 *   workspace >= pdec_grounding_workspace_size(dims) bytes, device, contents ignored.
 * Asynchronous on `stream` (two launches).  Returns a pdec_status.
 */
int pdec_segment_grounding(const pdec_ground_dims* dims, const void* g, const void* p, const int32_t* cu_seg,
                           float threshold, float* scores, uint8_t* salient, void* workspace,
                           size_t workspace_bytes, void* stream);

/*
 * Adaptive semantic aggregation into the global event tokens (§3.3,
 * "Adaptive Semantic Aggregation", strategies (1)-(3)).  For the K event
 * token embeddings g_i of a video and its N audio-visual prefix token
 * embeddings x_n, with the salient segments of each event (the output of
 * pdec_segment_grounding):
 *   out_i = g_i + sum_{n in sel_i} w_n x_n / sum_{n in sel_i} w_n,
 * sel_i the tokens of event i's salient segments; out_i = g_i when sel_i is
 * empty or its weights sum to 0.  The token weights are
 *   PDEC_AGGR_UNIFORM    w_n = 1 (mean pooling);
 *   PDEC_AGGR_LEARNED    w_n = scores[n] (the caller's scoring head);
 *   PDEC_AGGR_ATTENTION  the attention weights of the last text query token
 *                        over the tokens, averaged over its query heads:
 *                        w_n = (1/H_q) sum_h exp(scale <q_h, k[n, h / (H_q/H_kv)]> - lse[h]),
 *                        lse the log-normalisers of that token's attention rows
 *                        (the decode step's lse output for it).
 * Segments, clamping and determinism as for pdec_segment_grounding: sums run
 * in float32 in a fixed order (per 64-token chunk, per segment, per event),
 * and each output element is rounded once to bf16.
 */
enum { PDEC_AGGR_UNIFORM = 0, PDEC_AGGR_LEARNED = 1, PDEC_AGGR_ATTENTION = 2 };

typedef struct pdec_aggr_dims {
    int32_t num_events;    /* K >= 1                                                   */
    int32_t num_tokens;    /* N >= 1                                                   */
    int32_t num_segments;  /* S >= 1                                                   */
    int32_t hidden;        /* embedding width: a multiple of 8, at most 8192           */
    int32_t mode;          /* PDEC_AGGR_UNIFORM, PDEC_AGGR_LEARNED or PDEC_AGGR_ATTENTION */
    int32_t num_q_heads;   /* attention mode: H_q, 1..64, a multiple of num_kv_heads   */
    int32_t num_kv_heads;  /* attention mode: H_kv, divides num_q_heads                */
    int32_t head_dim;      /* attention mode: 64 or 128                                */
    float softmax_scale;   /* attention mode: 0 means 1/sqrt(head_dim)                 */
    int32_t dtype;         /* PDEC_DTYPE_BF16 (the only type with a kernel)            */
} pdec_aggr_dims;

/* Workspace bytes for pdec_aggregate (0 for invalid dims).  Host only. */
size_t pdec_aggregation_workspace_size(const pdec_aggr_dims* dims);

/*
 *   g [K, hidden], x [N, hidden]   device, bf16, rows contiguous, 16-byte aligned;
 *   cu_seg [S + 1] int32           device, non-decreasing from 0 to N (not checked:
 *                                  ranges are clamped to [0, N), so a bad table gives
 *                                  wrong sums, never a stray access);
 *   salient [K, S] uint8           device, nonzero = salient;
 *   scores [N] float32             device, learned mode only (else ignored, may be NULL);
 *   q [H_q, D], k [N, H_kv, D]     device, bf16, 16-byte aligned, attention mode only:
 *                                  the last text token's queries and the audio-visual
 *                                  tokens' keys (a contiguous slice of the prefix cache);
 *   lse [H_q] float32              device, attention mode only;
 *   weights [N] float32            device, attention mode: if not NULL, receives the
 *                                  token weights w_n; ignored in the other modes;
 *   out [K, hidden] bf16           device, written; may be g itself (in place);
 *   workspace >= pdec_aggregation_workspace_size(dims) bytes, device, 256-byte
 *                                  aligned, contents ignored.
 * Asynchronous on `stream` (three launches).
 * Returns a pdec_status.
 */
int pdec_aggregate(const pdec_aggr_dims* dims, const void* g, const void* x, const int32_t* cu_seg,
                   const uint8_t* salient, const float* scores, const void* q, const void* k, const float* lse,
                   float* weights, void* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward pass of the whole-branch attention (the training form of the §3.4
 * mask, as computed by pdec_attn_step with queries_per_stream N >= 1), for
 * one video.  Given the forward's out and lse and the gradient dout of a loss
 * with respect to out, for every live query row i (stream e with n_e > 0,
 * token j, head h) and every key k it sees (the prefix and its own rows
 * 0 .. min(j, n_e - 1)):
 *   p_ik = exp(scale <q_i, k_k> - lse_i),   D_i = <dout_i, out_i>,
 *   ds_ik = p_ik (<dout_i, v_k> - D_i),
 *   dq_i = scale sum_k ds_ik k_k,  dk_k = scale sum_i ds_ik q_i,  dv_k = sum_i p_ik dout_i.
 * Rows of ended streams add nothing; keys no row sees get 0.  With one stream
 * and no prefix (the prefix as the stream's rows) this is the backward of
 * plain causal attention.  dims as for pdec_attn_step: bf16, head_dim 64 or
 * 128, plan_mask 0 and cross_causal 0 (else PDEC_ERR_UNSUPPORTED).
 * P and ds meet the matrix cores in bf16, as the forward's P does; every
 * sum is float32.
 */
/* Workspace bytes for pdec_attn_prefill_backward (0 for invalid dims). Host only. */
size_t pdec_backward_workspace_size(const pdec_dims* dims);

/*
 *   q, out, dout [E, N, H_q, D]   device, bf16, 16-byte aligned;
 *   k_prefix, v_prefix [Lmax, H_kv, D], k_event, v_event [E, cap, H_kv, D]
 *                                 device, bf16, as for the forward call;
 *   event_lens [E], prefix_lens [1] device int32, as for the forward call;
 *   lse [E, N, H_q]               device, float32, the forward's lse;
 *   dq [E, N, H_q, D], dk_prefix, dv_prefix [Lmax, H_kv, D],
 *   dk_event, dv_event [E, cap, H_kv, D]
 *                                 device, float32, 16-byte aligned, every element written;
 *   workspace >= pdec_backward_workspace_size(dims) bytes, device.
 * Prefix pointers may be NULL when max_prefix_len is 0.  Asynchronous on
 * `stream` (three launches).  Returns a pdec_status.
 */
int pdec_attn_prefill_backward(const pdec_dims* dims, const void* q, const void* k_prefix, const void* v_prefix,
                               const void* k_event, const void* v_event, const int32_t* event_lens,
                               const int32_t* prefix_lens, const void* out, const float* lse, const void* dout,
                               float* dq, float* dk_prefix, float* dv_prefix, float* dk_event, float* dv_event,
                               void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* PDEC_H */
