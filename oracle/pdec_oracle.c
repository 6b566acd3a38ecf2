/*
 * Plain CPU oracle for the event-factorized parallel-decode attention step
 * (PadCaptioner, arXiv 2607.02963, §3.4 "Dependency-Restructured Parallel
 * Decoding", Eq. 3 and the attention mask it describes with Fig. 3).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg may load it.  It shares
 * no code, header, table or helper with the HIP library, and the HIP library
 * never calls it.
 *
 * What is computed (one decode step, one attention layer):
 *   A video has a prefix P of L tokens (audio-visual chunks, the instruction
 *   and the latent plan tokens G^1..G^K; §3.1, §3.3) and E event streams.
 *   Stream e owns a local cache of n_e rows: its anchor and the local tokens
 *   it has generated, the newest row being the token whose query is asked
 *   now.  Per §3.4 the query of stream e may see (1) every prefix token and
 *   (2) the rows of its own stream; rows of every other stream are masked.
 *   The oracle writes that rule out literally: it lays the keys out as one
 *   sequence U = [prefix | stream 0 rows | stream 1 rows | ...] (the
 *   full-sequence picture of Fig. 3), builds an explicit 0/1 mask over U, and
 *   evaluates ordinary softmax attention under that mask, two passes, fixed
 *   summation order.  No split, no online softmax, no blocking.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - n_e counts the stream's visible own rows including the current token
 *     (append first, then attend; the standard KV-cache convention).
 *   - n_e == 0 marks a stream that has ended (EOS, §3.4 last paragraph): it
 *     issues no query; its output row is 0 and its log-sum-exp is -inf.
 *   - scores are scale * <q, k>, scale = 1/sqrt(D) unless given.
 *   - grouped-query heads: query head h reads key/value head h / (H_q/H_kv).
 *   - lse is the natural-log log-sum-exp of the scaled scores.
 *   - the "self G-token only" variant of Table 8 (a branch sees, among the
 *     global plan tokens, only its own G^i) needs to know where the plan
 *     tokens are: the plan segment is taken as the last E*T prefix tokens,
 *     stream f's tokens being the f-th run of T of them (T tokens per
 *     stream, in stream order).
 *   - whole branches at once (oracle_attn_prefill, the training / prefill
 *     form): query j of a branch is the decode step of that branch at its
 *     token j, i.e. it sees its own rows 0 .. j (§3.4 pads branches to the
 *     longest with EOS when training; a branch with fewer rows stops there).
 *   - the rotary embedding at the shared step position (oracle_rope_append)
 *     is taken in the rotate-half form with frequencies theta^(-2i/D); a
 *     stream writing cache row t of video v stands at pos_base[v] + t.
 *
 * Arithmetic type: `real`, double by default.  The same source compiled with
 * -DORACLE_REAL=float gives the fp32 variant (functions suffixed _f32), used
 * only to measure the oracle's own rounding drift.  bf16 inputs are widened
 * exactly (a bf16 is the high half of an IEEE binary32).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef ORACLE_REAL
#define ORACLE_REAL double
#endif
typedef ORACLE_REAL real;

#define ORACLE_CAT2(a, b) a##_##b
#define ORACLE_CAT(a, b) ORACLE_CAT2(a, b)
#ifdef ORACLE_SUFFIX
#define ORACLE_FN(name) ORACLE_CAT(name, ORACLE_SUFFIX)
#else
#define ORACLE_FN(name) ORACLE_CAT(name, f64)
#endif

/* exp / log in the arithmetic type itself (float variant must not promote). */
static real r_exp(real x) { return sizeof(real) == sizeof(float) ? (real)expf((float)x) : (real)exp((double)x); }
static real r_log(real x) { return sizeof(real) == sizeof(float) ? (real)logf((float)x) : (real)log((double)x); }
static real r_cos(real x) { return sizeof(real) == sizeof(float) ? (real)cosf((float)x) : (real)cos((double)x); }
static real r_sin(real x) { return sizeof(real) == sizeof(float) ? (real)sinf((float)x) : (real)sin((double)x); }
static real r_pow(real x, real y) { return sizeof(real) == sizeof(float) ? (real)powf((float)x, (float)y) : (real)pow((double)x, (double)y); }

/* Element `idx` of a tensor stored as float32 (dtype 0) or bfloat16 (dtype 1). */
static real load_elem(const void* base, size_t idx, int dtype)
{
    if (dtype == 0) return (real)((const float*)base)[idx];
    uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (real)f;
}

/*
 * The §3.4 visibility rule for one video, as an explicit matrix.
 *   mask[e * U + j] = 1  iff  key j of the unified sequence is visible to the
 *   current query of stream e, with U = L + E * cap and
 *     j <  L                      : prefix token j              -> visible
 *     j =  L + f * cap + t        : row t of stream f's cache   -> visible
 *                                    iff f == e and t < n_e
 * Streams with n_e == 0 get an all-zero row (no query this step).
 * plan_mask != 0 with plan_T > 0 selects the "self G-token only" variant of
 * Table 8: prefix token j >= L - E*plan_T (the plan segment) is visible to
 * stream e only if it lies in e's own run of plan_T tokens.  The plan segment
 * must fit in the prefix (E*plan_T <= L).
 */
/* cross_limit > 0 (the "causal attention" row of Table 8, whole branches
 * only): row t of another stream f is also visible when t < cross_limit,
 * i.e. when its position comes before the query's. */
static int build_mask_x(int L, int E, int cap, const int32_t* n, int plan_mask, int plan_T, int cross_limit,
                        uint8_t* mask)
{
    if (L < 0 || E < 0 || cap < 0 || plan_T < 0 || (!mask && E > 0)) return -1;
    const long plan0 = (plan_mask && plan_T > 0) ? (long)L - (long)E * plan_T : (long)L;
    if (plan0 < 0) return -1;
    const long U = (long)L + (long)E * cap;
    for (int e = 0; e < E; ++e) {
        uint8_t* row = mask + (long)e * U;
        memset(row, 0, (size_t)U);
        if (n[e] <= 0) continue;
        for (long j = 0; j < L; ++j) row[j] = 1;                  /* shared prefix and plan tokens */
        for (long j = plan0; j < L; ++j) row[j] = (j - plan0) / plan_T == e; /* self G-token only */
        for (int f = 0; f < E; ++f)
            for (int t = 0; t < cap; ++t)
                if (f == e && t < n[e]) row[L + (long)f * cap + t] = 1; /* own stream only */
        for (int f = 0; f < E; ++f)                                            /* causal across streams */
            for (int t = 0; t < cap; ++t)
                if (f != e && t < n[f] && t < cross_limit) row[L + (long)f * cap + t] = 1;
    }
    return 0;
}

int ORACLE_FN(oracle_build_mask)(int L, int E, int cap, const int32_t* n, int plan_mask, int plan_T, uint8_t* mask)
{
    return build_mask_x(L, E, cap, n, plan_mask, plan_T, 0, mask);
}

/*
 * One decode step over a batch of videos.
 *
 *   num_videos            V
 *   cu_prefix[V+1]        video v owns prefix rows [cu_prefix[v], cu_prefix[v+1]) of k/v_prefix
 *   cu_events[V+1]        video v owns streams [cu_events[v], cu_events[v+1]) (rows of q/out/lse)
 *   H_q, H_kv, D          query heads, key/value heads (H_q % H_kv == 0), head dim
 *   cap                   rows per stream cache
 *   scale                 score scale (<= 0 selects 1/sqrt(D))
 *   dtype                 0: float32 tensors, 1: bfloat16 tensors (stored as uint16 bits)
 *   plan_mask, plan_T     0, 0: the full design; 1, T: "self G-token only" with T
 *                         plan tokens per stream (see oracle_build_mask)
 *   q        [SE, H_q, D]            SE = cu_events[V]
 *   k_prefix [SL, H_kv, D]           SL = cu_prefix[V]
 *   v_prefix [SL, H_kv, D]
 *   k_event  [SE, cap, H_kv, D]
 *   v_event  [SE, cap, H_kv, D]
 *   n        [SE]                    visible own rows per stream (0 = ended)
 *   row_select [SE * H_q] or NULL    compute only the selected (stream, head) rows
 *   out      [SE, H_q, D]  (real)    unselected rows are left untouched
 *   lse      [SE, H_q]     (real)
 *   probs    NULL, or for V == 1 a [SE, H_q, U] array that receives the
 *            attention weights over the unified key sequence (masked = 0)
 *   num_threads           0 = OpenMP default
 * Returns 0, or -1 on inconsistent arguments.
 */
static int attn_step_x(int num_videos, const int32_t* cu_prefix, const int32_t* cu_events, int H_q, int H_kv,
                       int D, int cap, double scale, int dtype, int plan_mask, int plan_T, int cross_limit,
                       const void* q, const void* k_prefix, const void* v_prefix, const void* k_event,
                       const void* v_event, const int32_t* n, const uint8_t* row_select, real* out, real* lse,
                       real* probs, int num_threads)
{
    if (num_videos < 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || D <= 0 || cap < 0) return -1;
    if (probs && num_videos != 1) return -1;
    const real tau = scale > 0 ? (real)scale : (real)(1.0 / sqrt((double)D));
    const int group = H_q / H_kv;
#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#else
    (void)num_threads;
#endif

    for (int v = 0; v < num_videos; ++v) {
        const int p0 = cu_prefix[v], L = cu_prefix[v + 1] - cu_prefix[v];
        const int e0 = cu_events[v], E = cu_events[v + 1] - cu_events[v];
        if (L < 0 || E < 0) return -1;
        for (int e = 0; e < E; ++e)
            if (n[e0 + e] < 0 || n[e0 + e] > cap) return -1;
        const long U = (long)L + (long)E * cap;
        uint8_t* mask = (uint8_t*)malloc((size_t)(E > 0 ? E : 1) * (size_t)(U > 0 ? U : 1));
        if (!mask) return -1;
        if (build_mask_x(L, E, cap, n + e0, plan_mask, plan_T, cross_limit, mask) != 0) {
            free(mask);
            return -1;
        }

        int bad = 0;
#pragma omp parallel for schedule(dynamic, 1)
        for (long row = 0; row < (long)E * H_q; ++row) {
            const int e = (int)(row / H_q), h = (int)(row % H_q);
            const long grow = (long)(e0 + e) * H_q + h; /* global (stream, head) row */
            if (row_select && !row_select[grow]) continue;
            const int g = h / group;
            real* o = out + grow * D;
            if (n[e0 + e] == 0) { /* ended stream: no query this step */
                for (int d = 0; d < D; ++d) o[d] = 0;
                lse[grow] = -(real)INFINITY;
                if (probs) for (long j = 0; j < U; ++j) probs[grow * U + j] = 0;
                continue;
            }
            real* s = (real*)malloc(sizeof(real) * (size_t)(U > 0 ? U : 1));
            if (!s) { bad = 1; continue; }
            const uint8_t* mrow = mask + (long)e * U;

            /* pass 1: scores of the visible keys, and their maximum */
            real m = -(real)INFINITY;
            for (long j = 0; j < U; ++j) {
                if (!mrow[j]) continue; /* masked keys are never read */
                size_t kbase;
                if (j < L) kbase = ((size_t)(p0 + j) * H_kv + g) * D;
                else {
                    const long f = (j - L) / cap, t = (j - L) % cap;
                    kbase = (((size_t)(e0 + f) * cap + t) * H_kv + g) * D;
                }
                const void* kt = j < L ? k_prefix : k_event;
                real dot = 0;
                for (int d = 0; d < D; ++d)
                    dot += load_elem(q, (size_t)grow * D + d, dtype) * load_elem(kt, kbase + d, dtype);
                s[j] = tau * dot;
                if (s[j] > m) m = s[j];
            }

            /* pass 2: normaliser, weighted sum of values, log-sum-exp */
            real l = 0;
            for (long j = 0; j < U; ++j)
                if (mrow[j]) l += r_exp(s[j] - m);
            for (int d = 0; d < D; ++d) o[d] = 0;
            for (long j = 0; j < U; ++j) {
                if (!mrow[j]) {
                    if (probs) probs[grow * U + j] = 0;
                    continue;
                }
                size_t vbase;
                if (j < L) vbase = ((size_t)(p0 + j) * H_kv + g) * D;
                else {
                    const long f = (j - L) / cap, t = (j - L) % cap;
                    vbase = (((size_t)(e0 + f) * cap + t) * H_kv + g) * D;
                }
                const void* vt = j < L ? v_prefix : v_event;
                const real p = r_exp(s[j] - m) / l;
                if (probs) probs[grow * U + j] = p;
                for (int d = 0; d < D; ++d) o[d] += p * load_elem(vt, vbase + d, dtype);
            }
            lse[grow] = m + r_log(l);
            free(s);
        }
        free(mask);
        if (bad) return -1;
    }
    return 0;
}

int ORACLE_FN(oracle_attn_step)(int num_videos, const int32_t* cu_prefix, const int32_t* cu_events,
                                int H_q, int H_kv, int D, int cap, double scale, int dtype,
                                int plan_mask, int plan_T, const void* q, const void* k_prefix, const void* v_prefix,
                                const void* k_event, const void* v_event, const int32_t* n,
                                const uint8_t* row_select, real* out, real* lse, real* probs,
                                int num_threads)
{
    return attn_step_x(num_videos, cu_prefix, cu_events, H_q, H_kv, D, cap, scale, dtype, plan_mask, plan_T, 0, q,
                       k_prefix, v_prefix, k_event, v_event, n, row_select, out, lse, probs, num_threads);
}

/*
 * Event-parallel decode loop for one video (§3.4: all streams step together;
 * a stream that has emitted EOS stops independently and the others go on).
 *
 * At step s (0 <= s < steps) stream e is live iff s < eos_step[e].  A live
 * stream first appends its new key/value row (k_new/v_new[s, e]) to its own
 * cache, so its visible row count becomes s + 1, then its query q[s, e]
 * attends.  A stream past its EOS step appends nothing and has n_e = 0.
 *
 *   k_prefix/v_prefix [L, H_kv, D];  q_steps [steps, E, H_q, D];
 *   k_new/v_new [steps, E, H_kv, D];  eos_step [E];  cap >= max live steps
 *   out [steps, E, H_q, D], lse [steps, E, H_q]  (real)
 */
int ORACLE_FN(oracle_decode_loop)(int steps, int E, int H_q, int H_kv, int D, int cap, int L,
                                  double scale, int dtype, const void* k_prefix, const void* v_prefix,
                                  const void* q_steps, const void* k_new, const void* v_new,
                                  const int32_t* eos_step, real* out, real* lse, int num_threads)
{
    if (steps < 0 || E <= 0 || cap <= 0 || L < 0) return -1;
    const size_t esz = dtype == 0 ? 4 : 2;
    const size_t row = (size_t)H_kv * D * esz;           /* one key/value row of one stream */
    unsigned char* kc = (unsigned char*)calloc((size_t)E * cap, row);
    unsigned char* vc = (unsigned char*)calloc((size_t)E * cap, row);
    int32_t* n = (int32_t*)calloc((size_t)E, sizeof(int32_t));
    int rc = (kc && vc && n) ? 0 : -1;
    const int32_t cu_prefix[2] = {0, L};
    const int32_t cu_events[2] = {0, E};
    for (int s = 0; s < steps && rc == 0; ++s) {
        for (int e = 0; e < E; ++e) {
            if (s < eos_step[e]) {
                if (n[e] >= cap) { rc = -1; break; }
                memcpy(kc + ((size_t)e * cap + n[e]) * row, (const unsigned char*)k_new + ((size_t)s * E + e) * row, row);
                memcpy(vc + ((size_t)e * cap + n[e]) * row, (const unsigned char*)v_new + ((size_t)s * E + e) * row, row);
                n[e] += 1;
            } else {
                n[e] = 0;
            }
        }
        if (rc) break;
        const unsigned char* qs = (const unsigned char*)q_steps + (size_t)s * E * H_q * D * esz;
        rc = ORACLE_FN(oracle_attn_step)(1, cu_prefix, cu_events, H_q, H_kv, D, cap, scale, dtype, 0, 0, qs,
                                         k_prefix, v_prefix, kc, vc, n, NULL,
                                         out + (size_t)s * E * H_q * D, lse + (size_t)s * E * H_q, NULL,
                                         num_threads);
    }
    free(kc);
    free(vc);
    free(n);
    return rc;
}

/*
 * Event-factorized attention over whole branches at once: the prefill /
 * training form of the §3.4 mask (the full-sequence picture of Fig. 3).
 * Stream e holds n_e rows of its own branch (§3.4 trains with the branches
 * padded by EOS to the longest, N); its query j, 0 <= j < N, sees every
 * prefix token and its own rows 0 .. min(j, n_e - 1), never another branch.
 * Query j of stream e is therefore the decode step of stream e holding
 * min(j + 1, n_e) rows, and the oracle evaluates exactly that, one step per
 * j.  A stream with n_e == 0 has no branch: its rows are 0 and -inf.
 * cross != 0 selects the "causal attention" row of Table 8 instead: the
 * tokens of one decoding step share a position (§3.4), and ordinary causal
 * attention then also shows query j every other branch's rows at earlier
 * positions, t < j (and t < n_f).
 *   q [SE, N, H_q, D];  out [SE, N, H_q, D], lse [SE, N, H_q]  (real);
 *   other arguments as for oracle_attn_step (no plan mask).
 */
int ORACLE_FN(oracle_attn_prefill)(int num_videos, const int32_t* cu_prefix, const int32_t* cu_events, int N,
                                   int cross, int H_q, int H_kv, int D, int cap, double scale, int dtype, const void* q,
                                   const void* k_prefix, const void* v_prefix, const void* k_event,
                                   const void* v_event, const int32_t* n, real* out, real* lse, int num_threads)
{
    if (num_videos < 1 || N < 1) return -1;
    const int SE = cu_events[num_videos];
    const size_t esz = dtype == 0 ? 4 : 2;
    const size_t qrow = (size_t)H_q * D * esz;  /* one query token, all heads */
    unsigned char* qj = (unsigned char*)malloc((size_t)SE * qrow + 1);
    int32_t* nj = (int32_t*)malloc((size_t)SE * sizeof(int32_t) + 4);
    real* oj = (real*)malloc((size_t)SE * H_q * D * sizeof(real) + 8);
    real* lj = (real*)malloc((size_t)SE * H_q * sizeof(real) + 8);
    int rc = (qj && nj && oj && lj) ? 0 : -1;
    for (int j = 0; j < N && rc == 0; ++j) {
        for (int e = 0; e < SE; ++e) {
            memcpy(qj + (size_t)e * qrow, (const unsigned char*)q + ((size_t)e * N + j) * qrow, qrow);
            nj[e] = n[e] <= 0 ? 0 : (j + 1 < n[e] ? j + 1 : n[e]);
        }
        rc = attn_step_x(num_videos, cu_prefix, cu_events, H_q, H_kv, D, cap, scale, dtype, 0, 0, cross ? j : 0, qj,
                         k_prefix, v_prefix, k_event, v_event, nj, NULL, oj, lj, NULL, num_threads);
        for (int e = 0; e < SE && rc == 0; ++e) {
            memcpy(out + ((size_t)e * N + j) * H_q * D, oj + (size_t)e * H_q * D, (size_t)H_q * D * sizeof(real));
            memcpy(lse + ((size_t)e * N + j) * H_q, lj + (size_t)e * H_q, (size_t)H_q * sizeof(real));
        }
    }
    free(qj);
    free(nj);
    free(oj);
    free(lj);
    return rc;
}

/*
 * Rotary position embedding at the shared decode position, with the cache
 * append it precedes (§3.4: tokens of all streams at one decoding step
 * carry one position index, so one rotation serves every stream of a
 * video at that step).
 *
 * Readings (the paper fixes the shared index, not the rotation, which is
 * its base model's):
 *   - rotate-half form: coordinate i of a head pairs with i + D/2 and turns
 *     by the angle pos * theta^(-2i/D), i < D/2:
 *       y[i]       = x[i] cos a - x[i + D/2] sin a
 *       y[i + D/2] = x[i + D/2] cos a + x[i] sin a
 *   - a stream of video v that writes its cache row t stands at position
 *     pos_base[v] + t; the live streams of a video step together, so they
 *     share it.
 *
 * For every stream e with live[e] != 0 and t = event_lens[e] < cap:
 *   q_rot[e, h] = R(pos) q[e, h] for every query head,
 *   k_rot[e, g] = R(pos) k_new[e, g] for every kv head,
 *   new_lens[e] = t + 1   (cache row t receives k_rot and v_new).
 * A stream with live[e] == 0 ends: new_lens[e] = 0, nothing rotated.  A live
 * stream whose cache is full keeps its count and is not rotated.  Rows not
 * rotated are left NaN in q_rot / k_rot.
 *   cu_events [V + 1]; pos_base [V]; q [SE, H_q, D]; k_new [SE, H_kv, D];
 *   q_rot [SE, H_q, D], k_rot [SE, H_kv, D] (real); lens in/out [SE].
 */
static void rotate_head(const void* x, size_t base, int D, int dtype, real pos, real theta, real* y)
{
    const int half = D / 2;
    for (int i = 0; i < half; ++i) {
        const real a = pos * r_pow(theta, -(real)(2 * i) / (real)D);
        const real c = r_cos(a), s = r_sin(a);
        const real x1 = load_elem(x, base + i, dtype);
        const real x2 = load_elem(x, base + i + half, dtype);
        y[i] = x1 * c - x2 * s;
        y[i + half] = x2 * c + x1 * s;
    }
}

int ORACLE_FN(oracle_rope_append)(int V, const int32_t* cu_events, const int32_t* pos_base, int H_q, int H_kv,
                                  int D, int cap, double theta, int dtype, const void* q, const void* k_new,
                                  const int32_t* event_lens, const int32_t* live, real* q_rot, real* k_rot,
                                  int32_t* new_lens)
{
    if (V < 1 || D < 2 || D % 2 != 0 || cap < 1 || !(theta > 0.0)) return -1;
    const int SE = cu_events[V];
    for (size_t i = 0; i < (size_t)SE * H_q * D; ++i) q_rot[i] = (real)NAN;
    for (size_t i = 0; i < (size_t)SE * H_kv * D; ++i) k_rot[i] = (real)NAN;
    for (int v = 0; v < V; ++v) {
        for (int e = cu_events[v]; e < cu_events[v + 1]; ++e) {
            const int t = event_lens[e];
            if (!live[e]) {
                new_lens[e] = 0;
                continue;
            }
            if (t < 0 || t >= cap) {
                new_lens[e] = t;
                continue;
            }
            const real pos = (real)pos_base[v] + (real)t;
            for (int h = 0; h < H_q; ++h)
                rotate_head(q, ((size_t)e * H_q + h) * D, D, dtype, pos, (real)theta, q_rot + ((size_t)e * H_q + h) * D);
            for (int g = 0; g < H_kv; ++g)
                rotate_head(k_new, ((size_t)e * H_kv + g) * D, D, dtype, pos, (real)theta,
                            k_rot + ((size_t)e * H_kv + g) * D);
            new_lens[e] = t + 1;
        }
    }
    return 0;
}

/* Threads OpenMP will use for a parallel region (1 without OpenMP). */
int ORACLE_FN(oracle_max_threads)(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
