// Matrix-core split pass (bf16).
//
// The prefix part of a step is a dense contraction: for one kv head, every
// query row of a video (R = E*G of them) against every key of the shared
// prefix (§3.4, Eq. 3).  One work-group takes one chunk of the virtual key
// sequence (prefix units, then each stream's own units; see pdec_common.h)
// for up to 256 rows, so each prefix K/V byte is fetched from HBM once and
// used by all of those rows; an own unit of stream f is used by f's rows
// only.
//
// Work-group: 8 or 16 waves = WR row waves x WK key groups.  Row wave rw owns NT
// 16-row tiles; key group kg owns a contiguous 64/WK-key slice of every
// 64-key stage (one unit).  Keys stream through a 3-stage LDS ring filled by
// global_load_lds_dwordx4 (direct HBM -> LDS DMA, 1 KB per wave
// instruction, no staging registers), two stages in flight while the
// third is consumed; the query rows arrive the same way, ahead of the first
// stages, so the first stage's products start once it has landed.  Each key row (D bf16) is stored as D/8 16-byte chunks
// permuted by an XOR of the key index, so the matrix-core operand reads below
// hit distinct LDS banks (the transposing V read takes 8 keys per 32-lane
// phase, so the V permutation differs over 8 consecutive keys).
//
// Per 32-key block, with v_mfma_f32_16x16x32_bf16 (D = A(16x32) B(32x16)):
//   S^T  = K  Q^T    A = K rows from LDS (16 keys x 32 d), B = Q^T (registers)
//   O^T += V^T P^T   A = V^T via ds_read_b64_tr_b16, B = P^T (registers)
// The S^T accumulator gives lane l the scores of query row l%16 for keys
// 4(l/16)..+3 of each 16-key tile, which is exactly a B operand of the second
// product once rounded to bf16, so P never leaves registers and O^T holds
// that query row in the same lane as its softmax state.  The transposing LDS
// read hands lane l the values of d = l%16 for four consecutive keys, which
// is the A operand of V^T with the same key order as P^T.
//
// Softmax in base 2 with the q scale folded into the exponent
// (p = 2^(s*c - m)).  Each row keeps a reference max m, raised only when that
// row's block max exceeds it by more than 8 (then its O and l are rescaled);
// otherwise p <= 2^8 and the final ratio is exact.  A row's arithmetic never
// depends on another row's values.  Keys past a unit's valid count, and own
// units of other streams, are masked to -inf; DMA reads are clamped to the
// unit's last valid key, so nothing outside it is ever fetched.
#pragma once

#include <type_traits>

#include "pdec_common.h"

namespace pdec {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;

__device__ inline f32x4_t mfma_16x16x32(bf16x8_t a, bf16x8_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8_t as_bf16x8(u32x4_t x) { return __builtin_bit_cast(bf16x8_t, x); }

typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// Two floats to a bf16 pair (round to nearest even), one v_cvt_pk_bf16_f32.
__device__ inline uint32_t pack_bf16x2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// Reduction over the 4 lane groups (lanes l, l^16, l^32, l^48) that hold one
// query row in the S^T accumulator layout.  v_permlane16_swap exchanges odd
// 16-lane rows of one operand with even rows of the other, v_permlane32_swap
// the upper half of one with the lower half of the other; with the value in
// both operands the two results hold the partner groups' values.  Plain VALU
// instructions: no LDS traffic.
__device__ inline float max_over_groups(float x)
{
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Initial reference max: finite, so no -inf special cases are needed; the
// first block with any visible key always re-references (its max exceeds
// this by more than 8), and 2^(s*c - kMinRef) is never evaluated before.
constexpr float kMinRef = -1e30f;


template <int D, int NT, int WR, int WK, bool MQ>
struct MfmaCfg {
    static constexpr int NW = WR * WK;            // waves
    static constexpr int KS = kUnit;              // keys per stage: one unit
    static constexpr int KW = KS / WK;            // keys per key group per stage
    // Ring slots.  A decode step keeps two stages in flight while the third
    // is consumed (a ring probe streams the decode layout as fast with two
    // stages in flight as with three or four) and stages its query rows by
    // DMA (QDMA); whole branches, whose items run many matrix-bound stages,
    // keep three in flight and load their query rows directly (measured
    // faster: the prefill call 649 against 700 us).
    static constexpr bool QDMA = !MQ;
    static constexpr int NSTAGE = QDMA ? 3 : 4;
    static constexpr int ROWB = D * 2;            // bytes per key row
    static constexpr int CH = D / 8;              // 16-byte chunks per key row
    static constexpr int STAGE_K = KS * ROWB;     // bytes of K per stage
    static constexpr int STAGE = 2 * STAGE_K;     // K then V
    static constexpr int KPI = 1024 / ROWB;       // keys per 1 KB DMA instruction
    static constexpr int DMA_PER_STAGE = STAGE / 1024;
    static constexpr int DMA_PER_WAVE = DMA_PER_STAGE / NW;
    static constexpr int KSTEPS = D / 32;
    static constexpr int DT = D / 16;
    static constexpr int RT = 16 * NT * WR;       // rows per item
    // V rows: chunk pairs XOR-permuted by the key, over 8 keys at D = 128 so
    // that the 8 keys one 32-lane phase of the transposing read touches fill
    // all banks (over 4 keys at D = 64, whose rows are half a bank period)
    static constexpr int VSW = D == 128 ? 14 : 6;
    static constexpr int LDS = NSTAGE * STAGE;
    // Query rows come in by DMA too (so that one in-order counter covers them
    // and the first stages): a wave's QB bytes land in the ring slot of stage
    // NSTAGE - 1, in the part that the wave's own DMA of that stage refills
    // (SR bytes), and the rest in an area of their own (XR bytes per wave).
    static constexpr int QB = NT * 16 * ROWB;
    static constexpr int SR = STAGE / NW;
    static constexpr int XR = QDMA ? QB - SR : 0;
    static constexpr int QX = NW * XR;
    static_assert(XR >= 0 && SR % 1024 == 0 && XR % 1024 == 0, "query staging");
    // A tail work-group's eight waves each stage a 32-key K and V block
    // (TVB bytes each) in the ring and then in qx, which is sized to hold the rest.
    static constexpr int TVB = 32 * ROWB;
    static constexpr int TAIL_LDS = 8 * 2 * TVB;
    static constexpr int QXA = QX > TAIL_LDS - LDS ? (QX > 1024 ? QX : 1024) : (TAIL_LDS - LDS > 1024 ? TAIL_LDS - LDS : 1024);
    static_assert(LDS % (2 * TVB) == 0, "a tail wave's buffers lie in one array");
    static_assert(NW == 8 || NW == 16, "eight or sixteen waves");
    static_assert(KW % 32 == 0, "key group slice is whole 32-key blocks");
    static_assert(DMA_PER_STAGE % NW == 0, "DMA split");
    // cross-key-group merge buffer fits in the ring
    static_assert(WK == 1 || (WR * NT * 16 * (D + 4) * 4 + 2 * WR * NT * 16 * 4) <= LDS, "merge buffer");
};

// Byte offset of 16-byte chunk `ch` of key `key` inside a stage's K or V area.
template <int D>
__device__ inline int k_off(int key, int ch) { return key * (2 * D) + 16 * (ch ^ (key % (D / 8))); }
template <int D>
__device__ inline int v_off(int key, int ch) { return key * (2 * D) + 16 * (ch ^ ((2 * key) & (D == 128 ? 14 : 6))); }

// Per-stream tail pass, one wave: the G (<= 16) query rows of stream e and
// kv head g (pair = e * H_kv + g) against the stream's own keys 0 .. n_e - 1
// (§3.4: a stream's own rows are seen by its own queries only), into slot 0
// of those rows.  The rows fill one 16-row tile; lanes of rows l16 >= G
// compute on zero queries and write nothing.  The keys go in 32-key blocks
// through the wave's own LDS area (buf: K then V, in the items' layouts),
// filled by DMA (cache rows from a scalar base and 32-bit lane offsets; a
// block holding a fused append's new row, key n_e - 1, takes per-lane
// addresses to read that row from k_new / v_new); the arithmetic is the
// items' (base-2 scores, a reference max raised by more than 8, bf16 P, the
// normaliser as a product with ones).
template <int D>
__device__ inline void tail_pair(const StepArgs& a, uint32_t buf, int pair)
{
    constexpr int ROWB = D * 2, CH = D / 8, KSTEPS = D / 32, DT = D / 16, KPI = 1024 / ROWB;
    constexpr int VSW = D == 128 ? 14 : 6;
    constexpr int TVB = 32 * ROWB, PIECES = TVB / 1024;
    const int lane = threadIdx.x & 63, l16 = lane & 15, lg = lane >> 4;
    const int e = pair / a.H_kv, g = pair - e * a.H_kv;
    const int n = stream_len(a, e);
    if (n <= 0) return;  // ended: the finish pass reads no slot of its rows
    const int an = a.k_new ? appended_row(a, e) : -1;
    const long kstride = (long)a.H_kv * D;  // elements between key rows of one head
    const uint16_t* kc = static_cast<const uint16_t*>(a.k_event) + ((long)e * a.cap * a.H_kv + g) * D;
    const uint16_t* vc = static_cast<const uint16_t*>(a.v_event) + ((long)e * a.cap * a.H_kv + g) * D;
    const long nrow = ((long)e * a.H_kv + g) * D;
    const uint16_t* kn = a.k_new ? static_cast<const uint16_t*>(a.k_new) + nrow : kc;
    const uint16_t* vn = a.k_new ? static_cast<const uint16_t*>(a.v_new) + nrow : vc;
    const uint32_t kstrideB = (uint32_t)(kstride * 2);
    const float c = a.qscale;
    typedef __attribute__((address_space(3))) unsigned char lds_uchar_t;
    const lds_uchar_t* const kbuf = reinterpret_cast<const lds_uchar_t*>((uintptr_t)buf);
    const lds_uchar_t* const vbuf = kbuf + TVB;

    // Q^T operands: tile row l16 is query head g*G + l16 of stream e
    const bool row_ok = l16 < a.G;
    bf16x8_t qf[KSTEPS];
    {
        const uint16_t* q = static_cast<const uint16_t*>(a.q) + ((long)e * a.H_q + g * a.G + (row_ok ? l16 : 0)) * D;
#pragma unroll
        for (int t = 0; t < KSTEPS; ++t) {
            const u32x4_t x = *reinterpret_cast<const u32x4_t*>(q + 32 * t + 8 * lg);
            qf[t] = as_bf16x8(row_ok ? x : u32x4_t{0u, 0u, 0u, 0u});
        }
    }
    // operand reads (the items' offsets): K key l16, chunk 4t + lg; V^T key
    // 4 lg + l16 / 4 (+16), d = 16 dt + 4 (l16 % 4) .. +3
    int koff[KSTEPS], voff[DT];
#pragma unroll
    for (int t = 0; t < KSTEPS; ++t) koff[t] = l16 * ROWB + 16 * ((4 * t + lg) ^ (l16 % CH));
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        const int key = 4 * lg + (l16 >> 2);
        const int ch = 2 * dt + ((l16 & 3) >> 1);
        voff[dt] = key * ROWB + 16 * (ch ^ ((2 * key) & VSW)) + 8 * (l16 & 1);
    }

    f32x4_t o[DT], lsum = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_ref = kMinRef;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const bf16x8_t ones = as_bf16x8(u32x4_t{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});

    // Piece i of a block: keys i*KPI + lane/CH, each lane one 16-byte chunk,
    // permuted as in the items' K and V areas (the K permutation repeats
    // every CH/KPI pieces, the V one every 2)
    constexpr int KREP = CH / KPI;
    uint32_t kcho[KREP], vcho[2];
#pragma unroll
    for (int i = 0; i < KREP; ++i) kcho[i] = 16 * ((lane % CH) ^ ((i * KPI + lane / CH) % CH));
#pragma unroll
    for (int i = 0; i < 2; ++i) vcho[i] = 16 * ((lane % CH) ^ ((2 * (i * KPI + lane / CH)) & VSW));
    for (int kb = 0; kb < n; kb += 32) {
        if (an >= kb && an < kb + 32) {
#pragma unroll
            for (int i = 0; i < PIECES; ++i) {
                const int key = i * KPI + lane / CH;
                const int kk = min(kb + key, n - 1);
                dma_16B(reinterpret_cast<const unsigned char*>(kk == an ? kn : kc + kk * kstride) + kcho[i % KREP],
                        buf + 1024 * i);
                dma_16B(reinterpret_cast<const unsigned char*>(kk == an ? vn : vc + kk * kstride) + vcho[i % 2],
                        buf + TVB + 1024 * i);
            }
        } else {
#pragma unroll
            for (int i = 0; i < PIECES; ++i) {
                const uint32_t row = (uint32_t)min(kb + i * KPI + lane / CH, n - 1) * kstrideB;
                dma_16B_sbase(kc, row + kcho[i % KREP], buf + 1024 * i);
                dma_16B_sbase(vc, row + vcho[i % 2], buf + TVB + 1024 * i);
            }
        }
        wave_wait_vmcnt<0>();

        f32x4_t s[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            s[kt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) {
                const bf16x8_t kf = as_bf16x8(
                    *reinterpret_cast<const __attribute__((address_space(3))) u32x4_t*>(kbuf + 16 * kt * ROWB + koff[t]));
                s[kt] = mfma_16x16x32(kf, qf[t], s[kt]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) s[kt][i] = kb + 16 * kt + 4 * lg + i >= n ? kNegInf : s[kt][i];
        }
        const float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                               fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
        if (__any(mx * c > m_ref + 8.f)) {
            const float mt = max_over_groups(mx) * c;
            const bool up = mt > m_ref + 8.f;
            const float alpha = up ? fast_exp2(m_ref - mt) : 1.f;
            m_ref = up ? mt : m_ref;
            lsum *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
        }
        float p[8];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int i = 0; i < 4; ++i) p[4 * kt + i] = fast_exp2(fmaf(s[kt][i], c, -m_ref));
        const bf16x8_t pf = as_bf16x8(u32x4_t{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                              pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])});
        lsum = mfma_16x16x32(ones, pf, lsum);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const lds_uchar_t* va = vbuf + voff[dt];
            const s16x4_t x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)va);
            const s16x4_t x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4_t*)(va + 16 * ROWB));
            const u32x2_t xa = __builtin_bit_cast(u32x2_t, x0);
            const u32x2_t xb = __builtin_bit_cast(u32x2_t, x1);
            o[dt] = mfma_16x16x32(as_bf16x8(u32x4_t{xa.x, xa.y, xb.x, xb.y}), pf, o[dt]);
        }
        // this block's LDS reads are done before the next block's DMA refills buf
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }

    if (!row_ok) return;
    const float l = lsum[0];
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const long slot = ((long)e * a.H_q + g * a.G + l16) * a.max_chunks;  // slot 0 of the row
    uint16_t* dst = static_cast<uint16_t*>(a.part_o) + slot * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        const f32x4_t v = o[dt];
        *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * lg) =
            make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
    }
    if (lg == 0) *reinterpret_cast<float2*>(a.part_ml + 2 * slot) = make_float2(m_ref, l);
}

template <int D, int NT, int WR, int WK, bool PLAN, bool MQ>
__global__ __launch_bounds__(64 * WR * WK) void split_mfma_kernel(StepArgs a)
{
    using C = MfmaCfg<D, NT, WR, WK, MQ>;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[C::LDS];
    __shared__ __attribute__((aligned(1024))) unsigned char qx[C::QXA];
    __shared__ int tab_start[kMaxStreamsPerVideo + 1];
    __shared__ int tab_nlen[kMaxStreamsPerVideo];
    __shared__ int s_total;

    if constexpr (!MQ) {
        // per-stream tail pass (decode steps only; the kernels of whole
        // branches carry none of its code): waves 0..7, one (stream, kv
        // head) pair each
        if ((int)blockIdx.x < a.tail_blocks) {
            const int w = threadIdx.x >> 6;
            const int pair = (int)blockIdx.x * 8 + w;
            if (w < 8 && pair < a.num_events * a.H_kv) {
                const int off = w * 2 * C::TVB;
                tail_pair<D>(a, off < C::LDS ? lds_u32(lds + off) : lds_u32(qx + (off - C::LDS)), pair);
            }
            return;
        }
    }

    // ---- which item; every branch below is uniform over the work-group ----
    const int item = item_of_block(a, (int)blockIdx.x - a.tail_blocks);
    if (item < 0) return;
    const ItemId id = item_id(a, item);
    const VideoInfo vi = video_info(a, id.v);
    const int R = vi.E * a.G * a.qps;
    const int row0 = id.rg * C::RT;
    if (row0 >= R) return;
    const int nrows = min(C::RT, R - row0);

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int l16 = lane & 15;
    const int lg = lane >> 4;
    const int rw = w % WR;
    const int kg = w / WR;
    const float c = a.qscale;

    const int upre = (vi.L + kUnit - 1) / kUnit;
    const int upc = a.unit_per_chunk;
    const int u0 = id.c * upc;
    const bool first_item = id.c == 0 && id.g == 0 && id.rg == 0;
    int u1 = u0 + upc;
    if (a.tail_blocks > 0) {
        // the tail pass holds the own units: prefix units only, the chunks
        // after the tail's slot
        if (first_item && tid == 0) a.video_chunks[id.v] = min(a.slot0 + (upre + upc - 1) / upc, a.max_chunks);
        u1 = min(u1, upre);
    } else if (u1 > upre || first_item) {  // reaches own units, or reports the chunk count
        if (w == 0) {
            const int own = build_unit_table(a, vi, tab_start, tab_nlen);
            if (lane == 0) s_total = upre + own;
        }
        lds_barrier();
        const int total = s_total;
        if (first_item && tid == 0) a.video_chunks[id.v] = min(max((total + upc - 1) / upc, 1), a.max_chunks);
        u1 = min(u1, total);
    }
    // fused append without a finish pass (one chunk): this item stores the
    // appended rows of its kv head (else the finish pass does)
    const bool app_store = a.k_new && a.max_chunks == 1 && id.c == 0 && id.rg == 0;
    if (u0 >= u1) {
        if (app_store) fused_append_store(a, vi, id.g, 2);
        return;
    }
    int nstages = u1 - u0;
    if constexpr (MQ) {
        // whole branches: rows of one stream f see none of the units after
        // f's unit holding their largest token (other streams' units are
        // hidden without the causal-attention variant).  The item still
        // writes its partial state, empty if no stage is left.
        const int per = a.G * a.qps;
        const int f = row0 / per;
        if (!a.cross && (row0 + nrows - 1) / per == f && u1 > upre) {
            const int tok_hi = ((row0 + nrows - 1) / a.G) % a.qps;
            nstages = max(0, min(nstages, upre + tab_start[f] + tok_hi / kUnit + 1 - u0));
        }
    }

    const uint16_t* __restrict__ kpre = static_cast<const uint16_t*>(a.k_prefix);
    const uint16_t* __restrict__ vpre = static_cast<const uint16_t*>(a.v_prefix);
    const uint16_t* __restrict__ kev = static_cast<const uint16_t*>(a.k_event);
    const uint16_t* __restrict__ vev = static_cast<const uint16_t*>(a.v_event);
    const long stride = (long)a.H_kv * D;

    // DMA of one stage (unit u0 + st): this wave's DMA_PER_WAVE 1 KB pieces,
    // all of K or all of V.  Piece p covers KPI keys of K (p < DMA_PER_STAGE/2)
    // or of V; lane l moves chunk (l % CH) ^ swizzle(key) of key (l / CH) of
    // the piece, so the piece lands in LDS already permuted.  A unit with fewer
    // than 64 valid keys clamps each lane's key to its last valid one.
    constexpr int PK_HALF = C::DMA_PER_STAGE / 2;
    const bool dma_v = w * C::DMA_PER_WAVE >= PK_HALF;
    const int pk0 = w * C::DMA_PER_WAVE - (dma_v ? PK_HALF : 0);
    const int strideB = (int)(stride * 2);
    auto issue_stage = [&](int st) {
        const UnitInfo ui = unit_info(a, vi, upre, tab_start, tab_nlen, id.g, u0 + st);
        const uint16_t* kb = (ui.stream < 0 ? kpre : kev) + ui.key_off;
        const uint16_t* vb = (ui.stream < 0 ? vpre : vev) + ui.key_off;
        const unsigned char* base = reinterpret_cast<const unsigned char*>(dma_v ? vb : kb);
        const uint32_t ldsb =
            lds_u32(lds + (st % C::NSTAGE) * C::STAGE + (dma_v ? C::STAGE_K : 0) + pk0 * 1024);
        const int clamp = ui.nk - 1;
        // fused append: a stream's appended row (the last valid key of its
        // last unit) comes from k_new / v_new instead of the cache
        const AppendedKey ak = appended_key(a, vi, ui, id.g, 2);
        if (ak.key >= 0) {
            const unsigned char* nrow = dma_v ? ak.vrow : ak.krow;
#pragma unroll
            for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
                const int key = (pk0 + i) * C::KPI + lane / C::CH;
                const int slot = lane % C::CH;
                const int ch = dma_v ? (slot ^ ((2 * key) & C::VSW)) : (slot ^ (key % C::CH));
                const int kk = min(key, clamp);
                dma_16B(kk == ak.key ? nrow + 16 * ch : base + kk * strideB + 16 * ch, ldsb + 1024 * i);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
            const int key = (pk0 + i) * C::KPI + lane / C::CH;
            const int slot = lane % C::CH;
            const int ch = dma_v ? (slot ^ ((2 * key) & C::VSW)) : (slot ^ (key % C::CH));
            const uint32_t off = (uint32_t)(min(key, clamp) * strideB + 16 * ch);
            dma_16B_sbase(base, off, ldsb + 1024 * i);
        }
    };

    // rows of this lane: 16*(rw*NT+nt) + l16 within the item, stream-major
    const int wrow0 = row0 + 16 * rw * NT;                // first video row of this wave
    const bool row_wave_active = 16 * rw * NT < nrows;

    // The wave's query rows go out first, then the first NSTAGE-1 stages, all
    // as DMA: one in-order counter then says when the rows and stage 0 have
    // landed, and the later stages keep streaming while stage 0 is consumed.
    // Local row r of the wave sits at byte r*ROWB of its staging area with
    // the K rows' chunk permutation: bytes below SR in ring slot NSTAGE-1
    // (the part this wave's own DMA of stage NSTAGE-1 refills, after the
    // rows are read), the rest in qx.  Rows past the item's last are fetched
    // from its first row and zeroed after the read.
    unsigned char* const qslot = lds + (C::NSTAGE - 1) * C::STAGE + w * C::SR;
    unsigned char* const qext = qx + w * C::XR;
    const bool q_dma = C::QDMA && row_wave_active && nstages > 0;
    if (q_dma) {
        const uint16_t* __restrict__ q = static_cast<const uint16_t*>(a.q);
#pragma unroll
        for (int j = 0; j < C::QB / 1024; ++j) {
            const int r = j * C::KPI + lane / C::CH;  // local row
            const int ir = 16 * rw * NT + r;          // row within the item
            const long qrow = row_qrow(a, vi, id.g, row0 + (ir < nrows ? ir : 0));
            const int ch = (lane % C::CH) ^ (r % C::CH);
            unsigned char* dst = j * 1024 < C::SR ? qslot + j * 1024 : qext + (j * 1024 - C::SR);
            dma_16B(q + qrow * D + 8 * ch, lds_u32(dst));
        }
    }
#pragma unroll
    for (int st = 0; st < C::NSTAGE - 1; ++st)
        if (st < nstages) issue_stage(st);

    int lane_stream[NT];
    int lane_tok[NT];  // query token of the row within its stream (whole branches; 0 otherwise)
    bf16x8_t qf[NT][C::KSTEPS];  // Q^T operands: q[row][32t + 8lg .. +7]
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int r = 16 * (rw * NT + nt) + l16;
        const bool ok = r < nrows;
        lane_stream[nt] = ok ? (row0 + r) / (a.G * a.qps) : -2;
        lane_tok[nt] = ok ? ((row0 + r) / a.G) % a.qps : 0;
        if constexpr (!C::QDMA) {
            // direct loads, awaited with every stage in flight (plain loads
            // and DMA share one counter and complete out of order)
            const uint16_t* __restrict__ q = static_cast<const uint16_t*>(a.q);
            const long base = ok ? (long)row_qrow(a, vi, id.g, row0 + r) * D : 0;
#pragma unroll
            for (int t = 0; t < C::KSTEPS; ++t) {
                u32x4_t x = {0u, 0u, 0u, 0u};
                if (ok) x = *reinterpret_cast<const u32x4_t*>(q + base + 32 * t + 8 * lg);
                qf[nt][t] = as_bf16x8(x);
            }
        }
    }
    if constexpr (!C::QDMA) wait_vmcnt<0>();

    // Whole branches: the range of query tokens and streams among this
    // wave's rows (uniform over the wave).  No row sees an own key above the
    // largest token, and an own unit that lies below the smallest token of a
    // wave whose rows all belong to its stream is seen whole by every row.
    int w_tok_lo = 0x7fffffff, w_tok_hi = -1, w_str_lo = 0x7fffffff, w_str_hi = -1;
    if constexpr (MQ) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            if (lane_stream[nt] >= 0) {
                w_tok_lo = min(w_tok_lo, lane_tok[nt]);
                w_tok_hi = max(w_tok_hi, lane_tok[nt]);
                w_str_lo = min(w_str_lo, lane_stream[nt]);
                w_str_hi = max(w_str_hi, lane_stream[nt]);
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            w_tok_lo = min(w_tok_lo, __shfl_xor(w_tok_lo, off));
            w_tok_hi = max(w_tok_hi, __shfl_xor(w_tok_hi, off));
            w_str_lo = min(w_str_lo, __shfl_xor(w_str_lo, off));
            w_str_hi = max(w_str_hi, __shfl_xor(w_str_hi, off));
        }
        w_tok_lo = __builtin_amdgcn_readfirstlane(w_tok_lo);
        w_tok_hi = __builtin_amdgcn_readfirstlane(w_tok_hi);
        w_str_lo = __builtin_amdgcn_readfirstlane(w_str_lo);
        w_str_hi = __builtin_amdgcn_readfirstlane(w_str_hi);
    }

    // The row normaliser is one more matrix product per block, ones^T P^T:
    // its accumulator holds the row sum of the block's bf16 P (the same P
    // that meets V) in each of a lane's four elements, in every lane group of
    // the row, which spares the vector ALUs the sum (they bound the loop).
    f32x4_t o[NT][C::DT], lsum[NT];
    float m_ref[NT], l_part[NT];
    const bf16x8_t ones = as_bf16x8(u32x4_t{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        m_ref[nt] = kMinRef;
        lsum[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) o[nt][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    // Per-lane LDS byte offsets of the operand reads, relative to the first
    // key of a 16-key group (the XOR swizzle depends on the lane only).
    //  K: key 16kt + l16, chunk 4t + lg.
    //  V: key 4lg + l16/4 (+16), d = 16dt + 4(l16 % 4) .. +3 (8 bytes).
    int koff[C::KSTEPS], voff[C::DT];
#pragma unroll
    for (int t = 0; t < C::KSTEPS; ++t) koff[t] = l16 * C::ROWB + 16 * ((4 * t + lg) ^ (l16 % C::CH));
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
        const int key = 4 * lg + (l16 >> 2);
        const int ch = 2 * dt + ((l16 & 3) >> 1);
        voff[dt] = key * C::ROWB + 16 * (ch ^ ((2 * key) & C::VSW)) + 8 * (l16 & 1);
    }

    // One 32-key block of this wave: S^T, online softmax, O^T += V^T P^T.
    // MASKED: keys past nk and keys owned by another stream (an own unit, or
    // a plan key under the self-only mask) are excluded; the unmasked form
    // serves every full prefix unit before the plan segment.
    auto block = [&](auto masked_tag, const unsigned char* kbuf, const unsigned char* vbuf, int kb,
                     const UnitInfo& ui) {
        constexpr bool MASKED = decltype(masked_tag)::value;
        f32x4_t s[2][NT];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) s[kt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < C::KSTEPS; ++t) {
                const bf16x8_t kf =
                    as_bf16x8(*reinterpret_cast<const u32x4_t*>(kbuf + (kb + 16 * kt) * C::ROWB + koff[t]));
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) s[kt][nt] = mfma_16x16x32(kf, qf[nt][t], s[kt][nt]);
            }
        }
        if constexpr (MASKED) {
            // a prefix unit reaching into the plan segment (self-only mask)
            bool plan_unit = false;
            if constexpr (PLAN) plan_unit = __builtin_amdgcn_readfirstlane(ui.stream < 0 && ui.k0 + kUnit > vi.plan0);
            if (plan_unit) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int kj = kb + 16 * kt + 4 * lg + i;
                        const bool kout = kj >= ui.nk;
#pragma unroll
                        for (int nt = 0; nt < NT; ++nt) {
                            const bool hide = kout | plan_key_hidden(a, vi, ui.k0 + kj, lane_stream[nt]);
                            s[kt][nt][i] = hide ? kNegInf : s[kt][nt][i];
                        }
                    }
            } else {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool kout = kb + 16 * kt + 4 * lg + i >= ui.nk;
#pragma unroll
                        for (int nt = 0; nt < NT; ++nt) {
                            bool hide;
                            if constexpr (MQ) {
                                // whole branches: query j sees its own rows 0 .. j; with the
                                // causal-attention variant also other streams' rows 0 .. j-1
                                const bool other = lane_stream[nt] != ui.stream;
                                const int lim = other ? (a.cross ? lane_tok[nt] - 1 : -1) : lane_tok[nt];
                                hide = kout || (ui.stream >= 0 && ui.k0 + kb + 16 * kt + 4 * lg + i > lim);
                            } else {
                                hide = kout || (ui.stream >= 0 && lane_stream[nt] != ui.stream);
                            }
                            if (hide) s[kt][nt][i] = kNegInf;
                        }
                    }
            }
        }
        // Rows whose block max rose by more than 8 re-reference.  The test
        // takes each lane's own max: no lane above the threshold means no row
        // above it, so the max over a row's four lane groups is formed only
        // when some row may move (it is the same in all four groups, which
        // keeps a row's reference identical across them).
        float mx[NT];
        bool need = false;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            mx[nt] = fmaxf(fmaxf(fmaxf(s[0][nt][0], s[0][nt][1]), fmaxf(s[0][nt][2], s[0][nt][3])),
                           fmaxf(fmaxf(s[1][nt][0], s[1][nt][1]), fmaxf(s[1][nt][2], s[1][nt][3])));
            need |= mx[nt] * c > m_ref[nt] + 8.f;
        }
        if (__any(need)) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const float mt = max_over_groups(mx[nt]) * c;
                const bool up = mt > m_ref[nt] + 8.f;
                const float alpha = up ? fast_exp2(m_ref[nt] - mt) : 1.f;
                m_ref[nt] = up ? mt : m_ref[nt];
                lsum[nt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < C::DT; ++dt) o[nt][dt] *= alpha;
            }
        }
        bf16x8_t pf[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            float p[8];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) p[4 * kt + i] = fast_exp2(fmaf(s[kt][nt][i], c, -m_ref[nt]));
            const u32x4_t pk = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                                pack_bf16x2(p[6], p[7])};
            pf[nt] = as_bf16x8(pk);
            lsum[nt] = mfma_16x16x32(ones, pf[nt], lsum[nt]);
        }
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt) {
            const unsigned char* va = vbuf + kb * C::ROWB + voff[dt];
            const s16x4_t x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)va);
            const s16x4_t x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4_t*)(va + 16 * C::ROWB));
            const u32x2_t xa = __builtin_bit_cast(u32x2_t, x0);
            const u32x2_t xb = __builtin_bit_cast(u32x2_t, x1);
            const bf16x8_t vf = as_bf16x8(u32x4_t{xa.x, xa.y, xb.x, xb.y});
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) o[nt][dt] = mfma_16x16x32(vf, pf[nt], o[nt][dt]);
        }
    };

    for (int st = 0; st < nstages; ++st) {
        // after the barrier every wave's pieces of stage st have landed and
        // stage st-1 has been consumed, so its buffer can be refilled
        if (C::NSTAGE >= 4 && st + 2 < nstages) stage_barrier<2 * C::DMA_PER_WAVE>();
        else if (st + 1 < nstages) stage_barrier<C::DMA_PER_WAVE>();
        else stage_barrier<0>();
        if (C::QDMA && st == 0) {
            // the wave's query rows have landed (they precede stage 0 on its
            // counter): read the Q^T operands before this wave's DMA below
            // refills their part of the ring
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const bool ok = q_dma && 16 * (rw * NT + nt) + l16 < nrows;
#pragma unroll
                for (int t = 0; t < C::KSTEPS; ++t) {
                    const int off = nt * 16 * C::ROWB + koff[t];
                    const unsigned char* src = off < C::SR ? qslot + off : qext + (off - C::SR);
                    u32x4_t x = {0u, 0u, 0u, 0u};
                    if (q_dma) x = *reinterpret_cast<const u32x4_t*>(src);
                    qf[nt][t] = as_bf16x8(ok ? x : u32x4_t{0u, 0u, 0u, 0u});
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        }
        if (st + C::NSTAGE - 1 < nstages) issue_stage(st + C::NSTAGE - 1);

        const UnitInfo ui = unit_info(a, vi, upre, tab_start, tab_nlen, id.g, u0 + st);
        // an own unit of stream f only concerns the rows of f
        bool wave_has_rows = row_wave_active;
        if (ui.stream >= 0 && !(MQ && a.cross)) {
            const int f0 = ui.stream * a.G * a.qps, f1 = f0 + a.G * a.qps;  // video rows of stream f
            wave_has_rows = wave_has_rows && f0 < wrow0 + 16 * NT && f1 > wrow0;
        }
        bool whole = ui.stream < 0 && ui.nk == kUnit && (!PLAN || ui.k0 + kUnit <= vi.plan0);
        if constexpr (MQ) {
            if (ui.stream >= 0) {
                // own keys t are seen at most by rows whose token is >= t
                if (ui.k0 > w_tok_hi) wave_has_rows = false;
                whole = ui.nk == kUnit && w_str_lo == ui.stream && w_str_hi == ui.stream &&
                        ui.k0 + kUnit - 1 <= w_tok_lo;
            }
        }
        const unsigned char* kbuf = lds + (st % C::NSTAGE) * C::STAGE;
        const unsigned char* vbuf = kbuf + C::STAGE_K;
        if (wave_has_rows) {
            if (whole) {
#pragma unroll
                for (int b = 0; b < C::KW / 32; ++b) block(std::false_type{}, kbuf, vbuf, kg * C::KW + 32 * b, ui);
            } else {
#pragma unroll
                for (int b = 0; b < C::KW / 32; ++b) {
                    const int kb = kg * C::KW + 32 * b;
                    if (kb < ui.nk) block(std::true_type{}, kbuf, vbuf, kb, ui);
                }
            }
        }
    }

    if (app_store) fused_append_store(a, vi, id.g, 2);  // every DMA has landed

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) l_part[nt] = lsum[nt][0];

    if constexpr (WK == 2) {
        // key group 1 hands its state to key group 0 through LDS
        constexpr int OROW = D + 4;
        constexpr int RW_ROWS = NT * 16;
        float* obuf = reinterpret_cast<float*>(lds);
        float* mbuf = obuf + WR * RW_ROWS * OROW;
        float* lbuf = mbuf + WR * RW_ROWS;
        __syncthreads();  // ring no longer read; every DMA has landed
        if (kg == 1 && row_wave_active) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = rw * RW_ROWS + 16 * nt + l16;
#pragma unroll
                for (int dt = 0; dt < C::DT; ++dt)
                    *reinterpret_cast<f32x4_t*>(obuf + r * OROW + 16 * dt + 4 * lg) = o[nt][dt];
                if (lg == 0) {
                    mbuf[r] = m_ref[nt];
                    lbuf[r] = l_part[nt];
                }
            }
        }
        __syncthreads();
        if (kg == 1) return;
        if (row_wave_active) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int r = rw * RW_ROWS + 16 * nt + l16;
                const float m1 = mbuf[r], l1 = lbuf[r];
                const float M = fmaxf(m_ref[nt], m1);
                const float f0 = fast_exp2(m_ref[nt] - M);
                const float f1 = fast_exp2(m1 - M);
                l_part[nt] = f0 * l_part[nt] + f1 * l1;
                m_ref[nt] = M;
#pragma unroll
                for (int dt = 0; dt < C::DT; ++dt)
                    o[nt][dt] = f0 * o[nt][dt] + f1 * *reinterpret_cast<const f32x4_t*>(obuf + r * OROW + 16 * dt + 4 * lg);
            }
        }
    }

    if (!row_wave_active) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int r = 16 * (rw * NT + nt) + l16;
        if (r < nrows) {
            const long qr = row_qrow(a, vi, id.g, row0 + r);
            const long slot = qr * a.max_chunks + a.slot0 + id.c;
            // o / l in bf16: a convex combination of V rows, so in V's range
            const float inv = l_part[nt] > 0.f ? 1.f / l_part[nt] : 0.f;
            uint16_t* dst = static_cast<uint16_t*>(a.part_o) + slot * D;
            if (a.max_chunks == 1) {
                // A single chunk holds the whole row: the host launches no
                // finish pass, and the row's result is written here with the
                // finish's arithmetic for one slot (the same bf16 values and
                // lse), an ended stream giving 0 and -inf.
                const bool ended = stream_len(a, (int)(qr / ((long)a.H_q * a.qps))) <= 0;
                dst = static_cast<uint16_t*>(a.out) + qr * D;
#pragma unroll
                for (int dt = 0; dt < C::DT; ++dt) {
                    const f32x4_t v = o[nt][dt];
                    const uint2 val = make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
                    *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * lg) = ended ? make_uint2(0u, 0u) : val;
                }
                if (a.lse && lg == 0) a.lse[qr] = ended ? kNegInf : kLn2 * (m_ref[nt] + __log2f(l_part[nt]));
                continue;
            }
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                const f32x4_t v = o[nt][dt];
                *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * lg) =
                    make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
            }
            if (lg == 0) *reinterpret_cast<float2*>(a.part_ml + 2 * slot) = make_float2(m_ref[nt], l_part[nt]);
        }
    }
}

}  // namespace pdec
