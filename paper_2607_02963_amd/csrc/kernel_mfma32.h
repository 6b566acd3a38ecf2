// Matrix-core split pass of the decode step on 32-row tiles (bf16, D = 128,
// more than 64 query rows per kv head).
//
// Same work as split_mfma_kernel (kernel_mfma.h): one work-group takes one
// chunk of the virtual key sequence (prefix units, then each stream's own
// units; pdec_common.h) for up to 256 query rows of one (video, kv head), so
// each prefix K/V byte is fetched from HBM once for all of those rows (§3.4,
// Eq. 3), and leaves one partial softmax state per row.  What differs is the
// tile: every product is a v_mfma_f32_32x32x16_bf16 (D = A(32x16) B(16x32)),
// and a wave owns 32 query rows.  A K or V operand read from LDS then serves
// 32 rows instead of 16, so a 224-row item reads each staged key 7 times
// rather than 14, and a query row lives in two lanes (l and l ^ 32) rather
// than four.
//
// Work-group: 8 waves = WR row waves x WK key groups; row wave rw owns rows
// 32 rw .. 32 rw + 31 of the item, key group kg the 32-key blocks kg, kg + WK
// of every 64-key stage.  Keys stream through a 4-stage LDS ring filled by
// global_load_lds_dwordx4 (1 KB per wave instruction, no staging registers),
// three stages in flight while the fourth is consumed.  A key row's 16-byte
// chunks are XOR-permuted by the key so that both operand reads below hit
// distinct banks: chunk c of a K row sits at c ^ (key mod 16); of a V row at
// c ^ f(key mod 4), f = {0, 6, 12, 10}, which gives the 4 keys x 4 chunks one
// 32-lane phase of the transposing read touches (and the 4 x 2 of a 16-lane
// phase) distinct banks.
//
// Per 32-key block:
//   S^T  = K Q^T     A = K (32 keys x 16 d) from LDS: lane l reads key l%32,
//                    d 16ks + 8(l/32) .. +7; B = Q^T held in registers.
//   O^T += V^T P^T   A = V^T (32 d x 16 keys) from two ds_read_b64_tr_b16;
//                    B = P^T straight from the S^T accumulator.
// The S^T accumulator gives lane l, register i, the score of query row l%32
// and key 8(i/4) + 4(l/32) + i%4.  Registers 8j .. 8j+7 rounded to bf16 are
// the B operand of the j-th 16-key product, with its k slots 0..7 (lanes
// l < 32) holding keys 16j + {0..3, 8..11} and slots 8..15 keys 16j +
// {4..7, 12..15}; the transposing read, in which each 16-lane group turns
// four 4-element row pieces into one column per lane, hands the A operand the
// same keys in the same order (lanes of group q address keys 16j + 8r +
// 4(q/2) + 0..3, read r = 0, 1).  P never leaves registers.
//
// Softmax as in kernel_mfma.h: base 2 with the q scale folded into the
// exponent, a per-row reference max raised only when a block's max exceeds it
// by more than 8.  The row normaliser sums the bf16 P (the values that meet
// V) with v_dot2_f32_bf16, two keys per instruction; the two lanes of a row
// add their sums at the end.  Masking: keys past a unit's valid count, own
// units of other streams and (self-only plan mask) other streams' plan keys
// are set to -inf; DMA reads are clamped to the unit's last valid key.
#pragma once

#include "kernel_mfma.h"

namespace pdec {

typedef __attribute__((ext_vector_type(16))) float f32x16_t;

__device__ inline f32x16_t mfma_32x32x16(bf16x8_t a, bf16x8_t b, f32x16_t c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Sum of a row's value over its two lanes (l, l ^ 32), in every lane.
__device__ inline float sum_pair(float x)
{
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ inline float max_pair(float x)
{
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// acc + lo(x) + hi(x) with x a packed bf16 pair, products with 1.0 exact.
__device__ inline float add_bf16_pair(float acc, uint32_t x)
{
    typedef __attribute__((ext_vector_type(2))) __bf16 bf2;
    const bf2 one = {(__bf16)1.0f, (__bf16)1.0f};
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, x), one, acc, false);
}

// Chunk permutation of a V row (key mod 4 -> XOR mask), see above.
__device__ inline int m32_vswz(int key)
{
    const int k = key & 3;
    return (6 * (k & 1)) ^ (12 * (k >> 1));
}

// Where one wave's DMA pieces of unit u go (see split_m32_kernel): the
// unit's first key row of the wave's tensor (K for waves 0..3, V for 4..7),
// the LDS address of its first piece, the unit's valid keys and the number of
// the wave's pieces that hold any of them.  n = 0 past the item's last unit.
struct M32Pending {
    const unsigned char* base;
    uint32_t lds;
    int nk;
    int n;
};
__device__ inline M32Pending m32_pending(const StepArgs& a, const VideoInfo& vi, int upre, const int* start,
                                         const int* nlen, int g, int u, bool valid, bool is_v, int pk0,
                                         uint32_t lds_addr, int pieces, int keys_per_piece)
{
    M32Pending pd{nullptr, 0u, 0, 0};
    if (!valid) return pd;
    const UnitInfo ui = unit_info(a, vi, upre, start, nlen, g, u);
    const void* t = is_v ? (ui.stream < 0 ? a.v_prefix : a.v_event) : (ui.stream < 0 ? a.k_prefix : a.k_event);
    pd.base = static_cast<const unsigned char*>(t) + ui.key_off * 2;
    pd.lds = lds_addr;
    pd.nk = ui.nk;
    pd.n = min(pieces, max(0, (ui.nk + keys_per_piece - 1) / keys_per_piece - pk0));
    return pd;
}

template <int WR, int WK, bool PLAN>
__global__ __launch_bounds__(512) void split_m32_kernel(StepArgs a)
{
    constexpr int D = 128;
    constexpr int NW = 8;
    static_assert(WR * WK == NW, "eight waves");
    static_assert(WK == 1 || WK == 2, "one or two key groups");
    constexpr int NSTAGE = 4;
    constexpr int ROWB = D * 2;                  // bytes per key row
    constexpr int CH = D / 8;                    // 16-byte chunks per key row
    constexpr int STAGE_K = kUnit * ROWB;        // K bytes of one 64-key stage
    constexpr int STAGE = 2 * STAGE_K;           // K then V
    constexpr int KPI = 1024 / ROWB;             // keys per 1 KB DMA instruction
    constexpr int DMA_PER_STAGE = STAGE / 1024;
    constexpr int DMA_PER_WAVE = DMA_PER_STAGE / NW;
    constexpr int RT = 32 * WR;                  // rows per item
    constexpr int NB = 2 / WK;                   // 32-key blocks per wave and stage
    constexpr int OROW = D + 4;                  // floats per row of the key-group merge buffer
    static_assert(WK == 1 || RT * OROW * 4 + 2 * RT * 4 <= NSTAGE * STAGE, "merge buffer fits the ring");

    __shared__ __attribute__((aligned(1024))) unsigned char lds[NSTAGE * STAGE];
    __shared__ int tab_start[kMaxStreamsPerVideo + 1];
    __shared__ int tab_nlen[kMaxStreamsPerVideo];
    __shared__ int s_total;

    // ---- which item; every branch below is uniform over the work-group ----
    const int item = item_of_block(a, blockIdx.x);
    if (item < 0) return;
    const ItemId id = item_id(a, item);
    const VideoInfo vi = video_info(a, id.v);
    const int R = vi.E * a.G;
    const int row0 = id.rg * RT;
    if (row0 >= R) return;
    const int nrows = min(RT, R - row0);

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int l32 = lane & 31;
    const int hi = lane >> 5;
    const int rw = w % WR;
    const int kg = w / WR;
    const float c = a.qscale;

    const int upre = (vi.L + kUnit - 1) / kUnit;
    const int upc = a.unit_per_chunk;
    const int u0 = id.c * upc;
    const bool first_item = id.c == 0 && id.g == 0 && id.rg == 0;
    int u1 = u0 + upc;
    if (u1 > upre || first_item) {  // reaches own units, or reports the chunk count
        if (w == 0) {
            const int own = build_unit_table(a, vi, tab_start, tab_nlen);
            if (lane == 0) s_total = upre + own;
        }
        lds_barrier();
        const int total = s_total;
        if (first_item && tid == 0) a.video_chunks[id.v] = min(max((total + upc - 1) / upc, 1), a.max_chunks);
        u1 = min(u1, total);
    }
    if (u0 >= u1) return;
    const int nstages = u1 - u0;

    const uint16_t* __restrict__ kpre = static_cast<const uint16_t*>(a.k_prefix);
    const uint16_t* __restrict__ vpre = static_cast<const uint16_t*>(a.v_prefix);
    const uint16_t* __restrict__ kev = static_cast<const uint16_t*>(a.k_event);
    const uint16_t* __restrict__ vev = static_cast<const uint16_t*>(a.v_event);
    const long stride = (long)a.H_kv * D;

    // the row of this lane: item row 32 rw + l%32, stream-major in the video
    const int wrow0 = 32 * rw;
    const bool row_wave_active = wrow0 < nrows;
    const int r_item = wrow0 + l32;
    const bool row_ok = r_item < nrows;
    const int my_stream = row_ok ? (row0 + r_item) / a.G : -2;
    bf16x8_t qf[8];  // Q^T operands, loaded after the first DMA stage is issued

    // DMA of one stage (unit u0 + st): DMA_PER_WAVE 1 KB pieces per wave,
    // four consecutive pieces of K (waves 0..3) or of V (waves 4..7).  Piece
    // p covers keys KPI p .. KPI p + KPI - 1 of the unit; lane l moves source
    // chunk (l % CH) ^ swizzle(key) of key (l / CH) of the piece, so the piece
    // lands in LDS already permuted.  A unit's keys are rows of H_kv * D
    // elements from its first key on, so a lane's byte offset within the unit
    // is fixed.  A partial unit (the last prefix unit, a stream's own rows)
    // issues only the pieces that hold valid keys; inside the last of them
    // keys past the end are clamped to the last valid key, so nothing outside
    // the unit is fetched.  The skipped rows keep older LDS contents (finite:
    // earlier K/V rows or the zeros written at the start), which the masking
    // hides.
    const uint32_t row_bytes = (uint32_t)(a.H_kv * D * 2);
    const bool w_is_v = w * DMA_PER_WAVE >= DMA_PER_STAGE / 2;
    const int pk0 = (w * DMA_PER_WAVE) % (DMA_PER_STAGE / 2);  // first piece of this wave in K or V
    uint32_t doff[DMA_PER_WAVE];
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) {
        const int key = (pk0 + i) * KPI + lane / CH;
        const int ch = (lane % CH) ^ (w_is_v ? m32_vswz(key) : (key % CH));
        doff[i] = key * row_bytes + 16 * ch;
    }
    using Pending = M32Pending;
    auto prep_stage = [&](int st) {
        return m32_pending(a, vi, upre, tab_start, tab_nlen, id.g, u0 + st, st < nstages, w_is_v, pk0,
                           lds_u32(lds + (st % NSTAGE) * STAGE + (w_is_v ? STAGE_K : 0) + pk0 * 1024),
                           DMA_PER_WAVE, KPI);
    };
    auto issue_piece = [&](const Pending& pd, int i) {
        if (i < pd.n) {
            const int key = (pk0 + i) * KPI + lane / CH;
            const uint32_t off = doff[i] - (uint32_t)max(0, key - (pd.nk - 1)) * row_bytes;
            dma_16B_sbase(pd.base, off, pd.lds + 1024 * i);
        }
    };
    // Wait until this wave's pieces of the current stage have landed (they
    // land in issue order, and n of its pieces of later stages were issued
    // after them) and its LDS operations are done, then barrier.  Waiting
    // for at most 8, 4 or 0 pieces in flight (n rounded down to one of them)
    // may wait for more than needed, never for less.
    auto barrier_pending = [&](int n) {
        if (n >= 8) stage_barrier<8>();
        else if (n >= 4) stage_barrier<4>();
        else stage_barrier<0>();
    };
    static_assert(DMA_PER_WAVE == 4, "a full stage is four pieces per wave");

    f32x16_t o[4];
    float m_ref = kMinRef, l_lane = 0.f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[dt][i] = 0.f;

    // Per-lane LDS byte offsets of the operand reads, relative to the first
    // key of a 32-key block.
    //  K, step ks: key l%32, chunk 2 ks + hi.
    //  V, d tile dt: key 4(q/2) + (l%16)/4 (+16 j + 8 r), d = 32 dt + 16(q%2) + 4(l%4) .. +3,
    //  q = l/16 the lane's 16-lane group.
    // K: chunk (2 ks + hi) ^ (l % 16) = 2 ks ^ (hi ^ l % 16), so step ks's
    // offset is koff0 ^ 32 ks (the row offset has no bits below 256).
    const int koff0 = l32 * ROWB + 16 * (hi ^ (lane & 15));
    int voff[4];
    {
        const int q = lane >> 4, i = lane & 15;
        const int key = 4 * (q >> 1) + (i >> 2);
#pragma unroll
        for (int dt = 0; dt < 4; ++dt) {
            const int ch = 4 * dt + 2 * (q & 1) + ((i & 3) >> 1);
            voff[dt] = key * ROWB + 16 * (ch ^ m32_vswz(key)) + 8 * (i & 1);
        }
    }

    auto read_k = [&](u32x4_t* kf, const unsigned char* kbuf) {
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) kf[ks] = *reinterpret_cast<const u32x4_t*>(kbuf + (koff0 ^ (32 * ks)));
    };
    auto scores_from = [&](const u32x4_t* kf) {
        f32x16_t s;
#pragma unroll
        for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) s = mfma_32x32x16(as_bf16x8(kf[ks]), qf[ks], s);
        return s;
    };

    // Masks block scores: keys at or past nk (kb = the block's first key in
    // the unit), own keys of another stream, plan keys of another stream.
    // Register i holds key kb + 4 hi + (8(i/4) + i%4): the lane part is
    // folded into the bounds, so each test compares a constant.
    auto mask = [&](f32x16_t& s, int kb, const UnitInfo& ui) {
        const bool other = ui.stream >= 0 && my_stream != ui.stream;
        const int lim = other ? -1 : ui.nk - kb - 4 * hi;  // registers with offset >= lim are hidden
        bool plan_unit = false;
        int plo = 0, phi = 0, pseg = 0;
        if constexpr (PLAN) {
            // plan keys j >= plan0 outside [lo, lo + T) are hidden; in register
            // offsets: >= pseg and outside [plo, phi)
            plan_unit = ui.stream < 0 && ui.k0 + kUnit > vi.plan0;
            const int j0 = ui.k0 + kb + 4 * hi;
            pseg = vi.plan0 - j0;
            plo = vi.plan0 + my_stream * a.plan_T - j0;
            phi = plo + a.plan_T;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int off = 8 * (i >> 2) + (i & 3);
            bool hide = off >= lim;
            if constexpr (PLAN) hide = hide | (plan_unit & (off >= pseg) & ((off < plo) | (off >= phi)));
            s[i] = hide ? kNegInf : s[i];
        }
    };

    // The 16 transposing reads of one block's V^T operands: read (j, dt, r)
    // at index 4 j + dt, r in the pair.
    auto read_v = [&](u32x4_t* vr, const unsigned char* vbuf) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) {
                const unsigned char* va = vbuf + (16 * j) * ROWB + voff[dt];
                const s16x4_t x0 =
                    __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)va);
                const s16x4_t x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4_t*)(va + 8 * ROWB));
                const u32x2_t xa = __builtin_bit_cast(u32x2_t, x0);
                const u32x2_t xb = __builtin_bit_cast(u32x2_t, x1);
                vr[4 * j + dt] = u32x4_t{xa.x, xa.y, xb.x, xb.y};
            }
    };

    // Lane max of a block's scores.
    auto lane_max = [&](const f32x16_t& s) {
        const float a0 = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
        const float a1 = fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7]));
        const float a2 = fmaxf(fmaxf(s[8], s[9]), fmaxf(s[10], s[11]));
        const float a3 = fmaxf(fmaxf(s[12], s[13]), fmaxf(s[14], s[15]));
        return fmaxf(fmaxf(a0, a1), fmaxf(a2, a3));
    };

    // Raises the reference max where a row's new max exceeds it by more than
    // 8.  Each lane tests its own max: no lane above the threshold means no
    // row above it; the row max over the lane pair (identical in both lanes,
    // so a row's reference stays identical) is formed only then.  Every
    // earlier block's P V product is already in O.
    auto rescale = [&](float mx) {
        if (__any(mx * c > m_ref + 8.f)) {
            const float mt = max_pair(mx) * c;
            const bool up = mt > m_ref + 8.f;
            const float alpha = up ? fast_exp2(m_ref - mt) : 1.f;
            m_ref = up ? mt : m_ref;
            l_lane *= alpha;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha;
        }
    };

    // P of one block in bf16 pairs (the B operands of its two 16-key
    // products), its sum added to the lane's normaliser.
    auto probs = [&](uint32_t* pk, const f32x16_t& s) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            pk[i] = pack_bf16x2(fast_exp2(fmaf(s[2 * i], c, -m_ref)), fast_exp2(fmaf(s[2 * i + 1], c, -m_ref)));
#pragma unroll
        for (int i = 0; i < 8; ++i) l_lane = add_bf16_pair(l_lane, pk[i]);
    };

    auto pv = [&](const uint32_t* pk, const u32x4_t* vr) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const bf16x8_t pf = as_bf16x8(u32x4_t{pk[4 * j], pk[4 * j + 1], pk[4 * j + 2], pk[4 * j + 3]});
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) o[dt] = mfma_32x32x16(as_bf16x8(vr[4 * j + dt]), pf, o[dt]);
        }
    };

    // One 32-key block with its masking: scores, softmax, O^T += V^T P^T.
    auto masked_block = [&](const unsigned char* kbuf, const unsigned char* vbuf, int kb, const UnitInfo& ui) {
        u32x4_t kf[8], vf[8];
        read_k(kf, kbuf);
        read_v(vf, vbuf);
        f32x16_t s = scores_from(kf);
        mask(s, kb, ui);
        rescale(lane_max(s));
        uint32_t pk[8];
        probs(pk, s);
        pv(pk, vf);
    };

    // Both 32-key blocks of a full prefix unit, in a fixed order (scheduling
    // barriers keep the compiler from regrouping it) that overlaps each
    // block's softmax with matrix-core work: block 0's scores; its rescale;
    // block 1's score products interleaved with block 0's exponentials;
    // block 1's new reference max (O is rescaled only after block 0's P V
    // products, which still use the old one); block 0's P V products
    // interleaved with block 1's exponentials; block 1's P V products.
    auto full_stage = [&](const unsigned char* kbuf, const unsigned char* vbuf, const Pending& pd) {
        u32x4_t kf[8], v0[8];
        read_k(kf, kbuf);
        read_v(v0, vbuf);
        __builtin_amdgcn_sched_barrier(0);
        f32x16_t s0, s1;
#pragma unroll
        for (int i = 0; i < 16; ++i) s0[i] = s1[i] = 0.f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            s0 = mfma_32x32x16(as_bf16x8(kf[ks]), qf[ks], s0);
            kf[ks] = *reinterpret_cast<const u32x4_t*>(kbuf + 32 * ROWB + (koff0 ^ (32 * ks)));
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        issue_piece(pd, 1);
        rescale(lane_max(s0));
        __builtin_amdgcn_sched_barrier(0);
        uint32_t p0[8], p1[8];
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) s1 = mfma_32x32x16(as_bf16x8(kf[ks]), qf[ks], s1);
        probs(p0, s0);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        // block 1's reference: decided now, applied to O after block 0's P V
        const float mx1 = lane_max(s1);
        float alpha1 = 1.f;
        const bool up1 = __any(mx1 * c > m_ref + 8.f);
        if (up1) {
            const float mt = max_pair(mx1) * c;
            const bool up = mt > m_ref + 8.f;
            alpha1 = up ? fast_exp2(m_ref - mt) : 1.f;
            m_ref = up ? mt : m_ref;
        }
        issue_piece(pd, 2);
        u32x4_t v1[8];
        read_v(v1, vbuf + 32 * ROWB);
        __builtin_amdgcn_sched_barrier(0);
        float l1 = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            p1[i] = pack_bf16x2(fast_exp2(fmaf(s1[2 * i], c, -m_ref)), fast_exp2(fmaf(s1[2 * i + 1], c, -m_ref)));
#pragma unroll
        for (int i = 0; i < 8; ++i) l1 = add_bf16_pair(l1, p1[i]);
        pv(p0, v0);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        issue_piece(pd, 3);
        if (up1) {
            l_lane *= alpha1;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt) o[dt] *= alpha1;
        }
        l_lane += l1;
        pv(p1, v1);
    };

    // Ring: stages 0..2 are issued up front; the barrier at the start of
    // stage st waits for st's pieces (every wave's) and finds stage st - 1
    // consumed, so its buffer takes stage st + 3.  An item that reaches a partial
    // unit first zeroes the V areas of the ring, so rows its DMA skips are
    // finite.
    if (u1 >= upre) {
#pragma unroll
        for (int b = 0; b < NSTAGE; ++b)
#pragma unroll
            for (int x = tid * 16; x < STAGE_K; x += 64 * NW * 16)
                *reinterpret_cast<u32x4_t*>(lds + b * STAGE + STAGE_K + x) = u32x4_t{0u, 0u, 0u, 0u};
        lds_barrier();
    }
    // Stage 0's DMA goes out before the query loads, so the two latencies
    // overlap; one wait covers both (the loads into LDS and into registers
    // are not counted in a common order), then stages 1 and 2 follow.
    {
        const Pending pd0 = prep_stage(0);
#pragma unroll
        for (int i = 0; i < DMA_PER_WAVE; ++i) issue_piece(pd0, i);
    }
    {  // Q^T operands (declared above): q[row][16 ks + 8 hi .. +7]
        const uint16_t* __restrict__ q = static_cast<const uint16_t*>(a.q);
        const long base = row_ok ? (long)row_qrow(a, vi, id.g, row0 + r_item) * D + 8 * hi : 0;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            u32x4_t x = {0u, 0u, 0u, 0u};
            if (row_ok) x = *reinterpret_cast<const u32x4_t*>(q + base + 16 * ks);
            qf[ks] = as_bf16x8(x);
        }
    }
    wait_vmcnt<0>();
    Pending pd1 = prep_stage(1), pd2 = prep_stage(2);
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) issue_piece(pd1, i);
#pragma unroll
    for (int i = 0; i < DMA_PER_WAVE; ++i) issue_piece(pd2, i);
    int n1 = pd1.n, n2 = pd2.n;  // this wave's pieces of the next two stages in flight

    for (int st = 0; st < nstages; ++st) {
        barrier_pending(n1 + n2);
        // stage st + 3's pieces: one now, the others between this stage's
        // products (a wave waits while the compute unit's address unit takes
        // its DMA, about 30 cycles per piece for all eight waves' pieces, so
        // pieces issued all at once hold every wave up)
        const Pending pd3 = prep_stage(st + NSTAGE - 1);
        issue_piece(pd3, 0);

        const UnitInfo ui = unit_info(a, vi, upre, tab_start, tab_nlen, id.g, u0 + st);
        // an own unit of stream f only concerns the rows of f
        bool wave_has_rows = row_wave_active;
        if (ui.stream >= 0) {
            const int f0 = ui.stream * a.G, f1 = f0 + a.G;  // video rows of stream f
            wave_has_rows = wave_has_rows && f0 < row0 + wrow0 + 32 && f1 > row0 + wrow0;
        }
        const bool whole = ui.stream < 0 && ui.nk == kUnit && (!PLAN || ui.k0 + kUnit <= vi.plan0);
        const unsigned char* kbuf = lds + (st % NSTAGE) * STAGE;
        const unsigned char* vbuf = kbuf + STAGE_K;
        if (wave_has_rows && whole && NB == 2) {
            full_stage(kbuf, vbuf, pd3);
        } else {
#pragma unroll
            for (int i = 1; i < DMA_PER_WAVE; ++i) issue_piece(pd3, i);
            if (wave_has_rows) {
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const int kb = 32 * (kg + WK * b);
                    if (kb < ui.nk) masked_block(kbuf + kb * ROWB, vbuf + kb * ROWB, kb, ui);
                }
            }
        }
        n1 = n2;
        n2 = pd3.n;
    }

    float l_row = sum_pair(l_lane);

    if constexpr (WK == 2) {
        // key group 1 hands its state to key group 0 through LDS; O^T element
        // (d, row) of register i of tile dt is d = 32 dt + 8(i/4) + 4 hi + i%4
        float* obuf = reinterpret_cast<float*>(lds);
        float* mbuf = obuf + RT * OROW;
        float* lbuf = mbuf + RT;
        __syncthreads();  // ring no longer read; every DMA has landed
        const int r = wrow0 + l32;
        if (kg == 1 && row_wave_active) {
#pragma unroll
            for (int dt = 0; dt < 4; ++dt)
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4)
                    *reinterpret_cast<f32x4_t*>(obuf + r * OROW + 32 * dt + 8 * g4 + 4 * hi) =
                        f32x4_t{o[dt][4 * g4], o[dt][4 * g4 + 1], o[dt][4 * g4 + 2], o[dt][4 * g4 + 3]};
            if (hi == 0) {
                mbuf[r] = m_ref;
                lbuf[r] = l_row;
            }
        }
        __syncthreads();
        if (kg == 1) return;
        if (row_wave_active) {
            const float m1 = mbuf[r], l1 = lbuf[r];
            const float M = fmaxf(m_ref, m1);
            const float f0 = fast_exp2(m_ref - M);
            const float f1 = fast_exp2(m1 - M);
            l_row = f0 * l_row + f1 * l1;
            m_ref = M;
#pragma unroll
            for (int dt = 0; dt < 4; ++dt)
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) {
                    const f32x4_t x = *reinterpret_cast<const f32x4_t*>(obuf + r * OROW + 32 * dt + 8 * g4 + 4 * hi);
#pragma unroll
                    for (int i = 0; i < 4; ++i) o[dt][4 * g4 + i] = f0 * o[dt][4 * g4 + i] + f1 * x[i];
                }
        }
    }

    if (!row_wave_active || !row_ok) return;
    const long qr = row_qrow(a, vi, id.g, row0 + r_item);
    const long slot = qr * a.max_chunks + id.c;
    // o / l in bf16: a convex combination of V rows, so in V's range
    const float inv = l_row > 0.f ? 1.f / l_row : 0.f;
    uint16_t* dst = static_cast<uint16_t*>(a.part_o) + slot * D;
    bool ended = false;
    if (a.max_chunks == 1) {
        // A single chunk holds the whole row: the host launches no finish
        // pass, and the row's result is written here with the finish's
        // arithmetic for one slot, an ended stream giving 0 and -inf.
        ended = a.event_lens[qr / a.H_q] <= 0;  // (no fused append reaches this kernel)
        dst = static_cast<uint16_t*>(a.out) + qr * D;
        if (a.lse && hi == 0) a.lse[qr] = ended ? kNegInf : kLn2 * (m_ref + __log2f(l_row));
    } else if (hi == 0) {
        *reinterpret_cast<float2*>(a.part_ml + 2 * slot) = make_float2(m_ref, l_row);
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const uint2 val = make_uint2(pack_bf16x2(o[dt][4 * g4] * inv, o[dt][4 * g4 + 1] * inv),
                                         pack_bf16x2(o[dt][4 * g4 + 2] * inv, o[dt][4 * g4 + 3] * inv));
            *reinterpret_cast<uint2*>(dst + 32 * dt + 8 * g4 + 4 * hi) = ended ? make_uint2(0u, 0u) : val;
        }
}

}  // namespace pdec
