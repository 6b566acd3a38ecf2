// Vector-ALU split pass: fewer query rows per kv head than one 16-row
// matrix-core tile (bf16), and every float32 step.
//
// Same work items as the matrix-core pass: (video, kv head, chunk of the
// virtual key sequence, row group of RT = 8 rows; pdec_common.h).  The
// work-group is 4 waves; wave w takes the chunk's units w, w+4, ... (64 keys
// each) with its own online-softmax state, and the four states are merged in
// LDS at the end.  Per unit, in both kernels:
//   softmax lane = key; the wave max of a row (DPP) is only formed when some
//           score exceeds the row's reference max by more than 8, which then
//           becomes that max (O and l rescaled), as in the matrix-core pass;
//   P V     lane = adjacent d, one coalesced V row per key load; the
//           probabilities are broadcast LDS reads.
// bf16 scores: a key row is split over LPK lanes of 32 bytes each (one pass
// covers 64/LPK keys); each lane keeps its 32-byte slice of the RT query
// rows in registers for the whole item and forms partial dot products
// through v_dot2c_f32_bf16 (exact products, float32 sums); the LPK partials
// of a key meet through DPP lane moves inside a 16-lane row and the key's RT
// scores go to LDS for the lane = key softmax.  The probabilities of keys
// 2j, 2j + 1 are rounded to bf16 and packed into one word, and P V takes two
// keys per v_dot2c_f32_bf16.  All K and V stays in registers, loaded one
// unit ahead of its use.
// float32 scores (the small-case precision path): lane = key, the key row in
// registers and the query rows in LDS, read as broadcasts.
// Keys past the unit's valid count, and for an own unit the rows of other
// streams, get probability 0; reads of keys past the valid count are clamped
// to the unit's last valid key, so nothing outside the unit is fetched.
#pragma once

#include <type_traits>

#include "pdec_common.h"

namespace pdec {

typedef __attribute__((ext_vector_type(2))) __bf16 valu_bf16x2_t;

// DPP lane move of a float over all rows (every source lane exists for the
// controls used with it), so the compiler can fold it into the consuming
// add or max.
template <int CTRL>
__device__ inline float dpp_f32(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, true));
}
// DPP lane move into the rows of ROW_MASK only; the other rows keep `old`.
template <int CTRL, int ROW_MASK>
__device__ inline float dpp_rows_f32(float old, float x)
{
    return __int_as_float(
        __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(x), CTRL, ROW_MASK, 0xf, false));
}
constexpr int kDppXor1 = 0xb1;        // quad_perm(1,0,3,2)
constexpr int kDppXor2 = 0x4e;        // quad_perm(2,3,0,1)
constexpr int kDppHalfMirror = 0x141; // lane i of 8 <- lane 7-i
constexpr int kDppMirror = 0x140;     // lane i of 16 <- lane 15-i
constexpr int kDppBcast15 = 0x142;    // row r+1 <- lane 15 of row r
constexpr int kDppBcast31 = 0x143;    // rows 2, 3 <- lane 31

// Sum over each aligned group of N lanes (N = 4, 8 or 16), every lane of the
// group left with the same value.
template <int N>
__device__ inline float group_sum(float x)
{
    static_assert(N == 4 || N == 8 || N == 16, "group size");
    x += dpp_f32<kDppXor1>(x);
    x += dpp_f32<kDppXor2>(x);
    if constexpr (N >= 8) x += dpp_f32<kDppHalfMirror>(x);
    if constexpr (N >= 16) x += dpp_f32<kDppMirror>(x);
    return x;
}

// Maximum over the 64 lanes, as a wave-uniform value.
__device__ inline float wave_max_uniform(float x)
{
    x = fmaxf(x, dpp_f32<kDppXor1>(x));
    x = fmaxf(x, dpp_f32<kDppXor2>(x));
    x = fmaxf(x, dpp_f32<kDppHalfMirror>(x));
    x = fmaxf(x, dpp_f32<kDppMirror>(x));
    x = fmaxf(x, dpp_rows_f32<kDppBcast15, 0xa>(x, x));
    x = fmaxf(x, dpp_rows_f32<kDppBcast31, 0xc>(x, x));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ inline float wave_sum_all(float x)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
    return x;
}

// Orders this wave's LDS accesses for the compiler; the hardware runs one
// wave's LDS instructions in issue order.
__device__ inline void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// a.lo * b.lo + a.hi * b.hi + c for bf16 pairs held as 32-bit words.
__device__ inline float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(valu_bf16x2_t, a), __builtin_bit_cast(valu_bf16x2_t, b),
                                           c, false);
}

// float -> bf16 bits, round to nearest even (finite inputs).
__device__ inline uint32_t bf16_bits_rne(float x)
{
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Unit description as wave-uniform (scalar) values: it is computed from LDS
// reads, which the compiler does not know to be the same in every lane.
__device__ inline UnitInfo uniform_unit(const UnitInfo& x)
{
    UnitInfo y;
    const uint64_t off = (uint64_t)x.key_off;
    y.key_off = (long)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(off >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)off));
    y.nk = __builtin_amdgcn_readfirstlane(x.nk);
    y.stream = __builtin_amdgcn_readfirstlane(x.stream);
    y.k0 = __builtin_amdgcn_readfirstlane(x.k0);
    return y;
}


// What every work item of the vector-ALU pass starts from.
struct ValuItem {
    ItemId id;
    VideoInfo vi;
    int nrows;  // rows of the item's group (1..RT)
    int row0;   // first row of the group within the video
    int upre;   // prefix units of the video
    int u0, u1; // the chunk's units [u0, u1)
};

// Item of this block; false when the block has nothing to do (uniform over
// the work-group).  Builds the per-video unit table in LDS when the chunk
// reaches past the prefix, and records the video's chunk count (first item).
template <int RT>
__device__ inline bool valu_item(const StepArgs& a, ValuItem& it, int* tab_start, int* tab_nlen, int* s_total)
{
    const int item = item_of_block(a, blockIdx.x);
    if (item < 0) return false;
    it.id = item_id(a, item);
    it.vi = video_info(a, it.id.v);
    const int R = it.vi.E * a.G;
    it.row0 = it.id.rg * RT;
    if (it.row0 >= R) return false;
    it.nrows = min(RT, R - it.row0);
    it.upre = (it.vi.L + kUnit - 1) / kUnit;
    const int upc = a.unit_per_chunk;
    it.u0 = it.id.c * upc;
    const bool first_item = it.id.c == 0 && it.id.g == 0 && it.id.rg == 0;
    it.u1 = it.u0 + upc;
    if (it.u1 > it.upre || first_item) {
        if (threadIdx.x < 64) {
            const int own = build_unit_table(a, it.vi, tab_start, tab_nlen);
            if (threadIdx.x == 0) *s_total = it.upre + own;
        }
        __syncthreads();
        const int total = *s_total;
        if (first_item && threadIdx.x == 0)
            a.video_chunks[it.id.v] = min(max((total + upc - 1) / upc, 1), a.max_chunks);
        it.u1 = min(it.u1, total);
    }
    return it.u0 < it.u1;
}

// Softmax of one row over the wave's 64 keys (lane = key): x is the scaled
// score or -inf.  Returns p = 2^(x - m_ref), raising m_ref (and rescaling
// l and the row's DPL output values) when some x exceeds it by more than 8.
template <int DPL>
__device__ inline float row_softmax(float x, float& m_ref, float& l_lane, float (&o_row)[DPL])
{
    if (__builtin_amdgcn_ballot_w64(x > m_ref + 8.f)) {  // rare after a row's first unit
        const float bm = wave_max_uniform(x);
        const float alpha = fast_exp2(m_ref - bm);
        m_ref = bm;
        l_lane *= alpha;
#pragma unroll
        for (int j = 0; j < DPL; ++j) o_row[j] *= alpha;
    }
    const float p = fast_exp2(x - m_ref);  // 0 for x = -inf
    l_lane += p;
    return p;
}

// Merge of the four waves' states of an item and the write of its slot.
// o0, o1, o2 hold waves 1, 2, 3's outputs (RT x D floats, row-major) in LDS;
// the lane owns d0 .. d0 + DPL - 1 when `owner`.
template <typename T, int D, int RT, int DPL>
__device__ inline void valu_merge_write(const StepArgs& a, const ValuItem& it, int w, int lane, bool owner, int d0,
                                        const float (&m_ref)[RT], const float (&l_lane)[RT], const float (&o)[RT][DPL],
                                        float (*m_s)[RT], float (*l_s)[RT], float* o0, float* o1, float* o2)
{
    constexpr int NW = 4;
    float* const o_other[3] = {o0, o1, o2};
    float lsum[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) lsum[r] = wave_sum_all(l_lane[r]);
    if (lane == 0) {
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            m_s[w][r] = m_ref[r];
            l_s[w][r] = lsum[r];
        }
    }
    if (w > 0 && owner) {
#pragma unroll
        for (int r = 0; r < RT; ++r)
#pragma unroll
            for (int j = 0; j < DPL; ++j) o_other[w - 1][r * D + d0 + j] = o[r][j];
    }
    __syncthreads();
    if (w != 0 || !owner) return;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        if (r >= it.nrows) break;
        float M = m_s[0][r];
#pragma unroll
        for (int x = 1; x < NW; ++x) M = fmaxf(M, m_s[x][r]);
        float f[NW];
        float L = 0.f;
#pragma unroll
        for (int x = 0; x < NW; ++x) {
            f[x] = fast_exp2(m_s[x][r] - M);  // 0 for a wave that saw none of the row's keys
            L += f[x] * l_s[x][r];
        }
        const long qr = row_qrow(a, it.vi, it.id.g, it.row0 + r);
        const long slot = qr * a.max_chunks + it.id.c;
        T* dst = static_cast<T*>(a.part_o) + slot * D + d0;
        const float inv = L > 0.f ? 1.f / L : 0.f;  // stored normalised, in the inputs' type
#pragma unroll
        for (int j = 0; j < DPL; ++j) {
            float acc = f[0] * o[r][j];
#pragma unroll
            for (int x = 1; x < NW; ++x) acc += f[x] * o_other[x - 1][r * D + d0 + j];
            dst[j] = from_f32<T>(acc * inv);
        }
        if (lane == 0) *reinterpret_cast<float2*>(a.part_ml + 2 * slot) = make_float2(M, L);
    }
}

// ----------------------------------------------------------------------------
// bf16: key rows split over lanes, everything in registers.
template <int D, int RT, bool PLAN>
__global__ __launch_bounds__(256) void split_valu_bf16_kernel(StepArgs a)
{
    constexpr int NW = 4;
    static_assert(RT == 8, "rows per item");
    static_assert(D == 64 || D == 128, "head dim");
    constexpr int ROWB = 2 * D;     // bytes per key row
    constexpr int LPK = ROWB / 32;  // lanes per key in the score pass (32 bytes each)
    constexpr int KPP = 64 / LPK;   // keys per score pass
    constexpr int NP = 64 / KPP;    // score passes per unit
    constexpr int DPL = D / 64;     // d per lane in P V

    __shared__ __attribute__((aligned(16))) float s_s[NW][64 * RT];     // scores [key][row]
    __shared__ __attribute__((aligned(16))) uint32_t p_s[NW][32 * RT];  // [key pair][row], packed bf16
    __shared__ __attribute__((aligned(16))) float o_s[NW - 1][RT * D];
    __shared__ float m_s[NW][RT], l_s[NW][RT];
    __shared__ int tab_start[kMaxStreamsPerVideo + 1];
    __shared__ int tab_nlen[kMaxStreamsPerVideo];
    __shared__ int s_total;

    ValuItem it;
    if (!valu_item<RT>(a, it, tab_start, tab_nlen, &s_total)) return;
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int lane = tid & 63;
    const float c = a.qscale;
    const uint32_t stride_b = (uint32_t)a.H_kv * ROWB;  // bytes between consecutive keys
    const int kslot = lane / LPK;                      // key of a score pass
    const int slice = lane % LPK;                      // 32-byte slice of the key row

    // this lane's slice of every query row (rows past nrows are 0)
    uint4 qx[RT][2];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const bool ok = r < it.nrows;  // wave-uniform
        const uint4* src = reinterpret_cast<const uint4*>(
            static_cast<const unsigned char*>(a.q) +
            (long)row_qrow(a, it.vi, it.id.g, it.row0 + min(r, it.nrows - 1)) * ROWB + slice * 32);
        const uint4 x0 = src[0], x1 = src[1];
        qx[r][0] = make_uint4(ok ? x0.x : 0u, ok ? x0.y : 0u, ok ? x0.z : 0u, ok ? x0.w : 0u);
        qx[r][1] = make_uint4(ok ? x1.x : 0u, ok ? x1.y : 0u, ok ? x1.z : 0u, ok ? x1.w : 0u);
    }
    int row_stream[RT];  // -2 past nrows; an own unit of stream f is seen by the rows of f only
#pragma unroll
    for (int r = 0; r < RT; ++r) row_stream[r] = r < it.nrows ? (it.row0 + r) / a.G : -2;
    float* const sw = s_s[w];
    uint32_t* const pw = p_s[w];

    auto k_base = [&](const UnitInfo& ui) {
        return static_cast<const unsigned char*>(ui.stream < 0 ? a.k_prefix : a.k_event) + ui.key_off * 2;
    };
    auto v_base = [&](const UnitInfo& ui) {
        return static_cast<const unsigned char*>(ui.stream < 0 ? a.v_prefix : a.v_event) + ui.key_off * 2;
    };
    // K: pass p gives lane (kslot, slice) key p*KPP + kslot, bytes slice*32 .. +32
    auto load_k = [&](const UnitInfo& ui, uint4 (&kx)[NP][2]) {
        const unsigned char* kb = k_base(ui);
        const AppendedKey ak = appended_key(a, it.vi, ui, it.id.g, 2);  // fused append: key from k_new
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int kk = min(p * KPP + kslot, ui.nk - 1);
            const uint32_t off = (uint32_t)kk * stride_b + (uint32_t)slice * 32u;
            const uint4* src = reinterpret_cast<const uint4*>(kk == ak.key ? ak.krow + slice * 32 : kb + off);
            kx[p][0] = src[0];
            kx[p][1] = src[1];
        }
    };
    // V: the lane's DPL adjacent d of every key, one coalesced row per key
    // (a uniform base per key and a fixed lane offset)
    const uint32_t v_lane = (uint32_t)lane * DPL * 2;
    auto load_v1 = [&](const unsigned char* base, uint32_t off) -> uint32_t {
        // a fresh 32-bit offset here, so the load takes the (SGPR base +
        // VGPR offset) form instead of a 64-bit address
        asm("" : "+v"(off));
        if constexpr (DPL == 2) return *reinterpret_cast<const uint32_t*>(base + off);
        else return *reinterpret_cast<const uint16_t*>(base + off);
    };
    auto load_v = [&](const UnitInfo& ui, uint32_t (&vw)[kUnit]) {
        const unsigned char* vb = v_base(ui);
        const AppendedKey ak = appended_key(a, it.vi, ui, it.id.g, 2);  // fused append: key from v_new
#pragma unroll
        for (int k = 0; k < kUnit; ++k) {
            const int kk = min(k, ui.nk - 1);
            vw[k] = load_v1(kk == ak.key ? ak.vrow : vb + (size_t)kk * stride_b, v_lane);
        }
    };

    float m_ref[RT], l_lane[RT], o[RT][DPL];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        m_ref[r] = -1e30f;  // finite: the first visible key always re-references
        l_lane[r] = 0.f;
#pragma unroll
        for (int j = 0; j < DPL; ++j) o[r][j] = 0.f;
    }

    // Loads run one unit ahead: the unit's K and V up front, the next unit's
    // K after this unit's scores and its V after this unit's P V.  The next
    // unit's loads are unconditional (a wave without one reloads its unit,
    // cached), so the compiler's load counting keeps them in flight.
    int u = it.u0 + w;
    if (u < it.u1) {
        UnitInfo ui = uniform_unit(unit_info(a, it.vi, it.upre, tab_start, tab_nlen, it.id.g, u));
        uint4 kx[NP][2];
        uint32_t vw[kUnit];
        load_k(ui, kx);
        __builtin_amdgcn_sched_barrier(0);
        load_v(ui, vw);
        for (;;) {
            const int nk = ui.nk;

            // ---- scores: KPP keys per pass, a key's RT scores to LDS ----
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                float sp[RT];
#pragma unroll
                for (int r = 0; r < RT; ++r) {
                    float x = 0.f;
                    x = dot2_bf16(qx[r][0].x, kx[p][0].x, x);
                    x = dot2_bf16(qx[r][0].y, kx[p][0].y, x);
                    x = dot2_bf16(qx[r][0].z, kx[p][0].z, x);
                    x = dot2_bf16(qx[r][0].w, kx[p][0].w, x);
                    x = dot2_bf16(qx[r][1].x, kx[p][1].x, x);
                    x = dot2_bf16(qx[r][1].y, kx[p][1].y, x);
                    x = dot2_bf16(qx[r][1].z, kx[p][1].z, x);
                    x = dot2_bf16(qx[r][1].w, kx[p][1].w, x);
                    sp[r] = group_sum<LPK>(x);
                }
                if (slice == 0) {
                    float* dst = sw + (p * KPP + kslot) * RT;
                    *reinterpret_cast<float4*>(dst) = make_float4(sp[0], sp[1], sp[2], sp[3]);
                    *reinterpret_cast<float4*>(dst + 4) = make_float4(sp[4], sp[5], sp[6], sp[7]);
                }
            }
            const int un = u + NW;
            const bool more = un < it.u1;  // wave-uniform
            const UnitInfo ui_next =
                more ? uniform_unit(unit_info(a, it.vi, it.upre, tab_start, tab_nlen, it.id.g, un)) : ui;
            load_k(ui_next, kx);  // kx is free since the scores
            wave_lds_sync();

            // ---- softmax per row, lane = key; P packed as bf16 pairs ----
            {
                const bool kvalid = lane < nk;
                const bool plan_unit = PLAN && ui.stream < 0 && ui.k0 + kUnit > it.vi.plan0;  // self-only mask
                const float4 x0 = *reinterpret_cast<const float4*>(sw + lane * RT);
                const float4 x1 = *reinterpret_cast<const float4*>(sw + lane * RT + 4);
                const float sx[RT] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
                uint32_t pv[RT];
#pragma unroll
                for (int r = 0; r < RT; ++r) {
                    bool row_sees = row_stream[r] != -2 && (ui.stream < 0 || row_stream[r] == ui.stream);
                    if (plan_unit) row_sees = row_sees & !plan_key_hidden(a, it.vi, ui.k0 + lane, row_stream[r]);
                    const float x = (kvalid && row_sees) ? sx[r] * c : kNegInf;
                    const float p = row_softmax<DPL>(x, m_ref[r], l_lane[r], o[r]);
                    const uint32_t bits = bf16_bits_rne(p);
                    const uint32_t nb = (uint32_t)__builtin_amdgcn_mov_dpp((int)bits, kDppXor1, 0xf, 0xf, true);
                    pv[r] = bits | (nb << 16);  // even lane: (key, key + 1)
                }
                if ((lane & 1) == 0) {
                    uint32_t* dst = pw + (lane >> 1) * RT;
                    *reinterpret_cast<uint4*>(dst) = make_uint4(pv[0], pv[1], pv[2], pv[3]);
                    *reinterpret_cast<uint4*>(dst + 4) = make_uint4(pv[4], pv[5], pv[6], pv[7]);
                }
            }
            wave_lds_sync();

            // ---- P V: lane = DPL adjacent d, two keys per dot ----
#pragma unroll
                for (int k = 0; k < kUnit; k += 2) {
                    if (k >= nk) continue;  // wave-uniform; keys past nk have p = 0
                    // (v_k[d], v_k+1[d]) for the lane's d
                    const uint32_t vj0 = __builtin_amdgcn_perm(vw[k + 1], vw[k], 0x05040100u);
                    const uint32_t vj1 = __builtin_amdgcn_perm(vw[k + 1], vw[k], 0x07060302u);
                    const uint32_t* pr = pw + (k >> 1) * RT;
                    const uint4 pa = *reinterpret_cast<const uint4*>(pr);
                    const uint4 pb = *reinterpret_cast<const uint4*>(pr + 4);
                    const uint32_t pp[RT] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
#pragma unroll
                    for (int r = 0; r < RT; ++r) {
                        o[r][0] = dot2_bf16(pp[r], vj0, o[r][0]);
                        if constexpr (DPL == 2) o[r][1] = dot2_bf16(pp[r], vj1, o[r][1]);
                    }
                }
            wave_lds_sync();  // s_s and p_s are rewritten by the next unit
            if (!more) break;
            load_v(ui_next, vw);  // vw is free again
            ui = ui_next;
            u = un;
        }
    }

    valu_merge_write<uint16_t, D, RT, DPL>(a, it, w, lane, true, lane * DPL, m_ref, l_lane, o, m_s, l_s, o_s[0], o_s[1],
                                 o_s[2]);
}

// ----------------------------------------------------------------------------
// float32, direct loads.
template <int D, int RT, bool PLAN>
__global__ __launch_bounds__(256) void split_valu_f32_kernel(StepArgs a)
{
    constexpr int NW = 4;
    static_assert(RT == 8, "rows per item");
    static_assert(D == 64 || D == 128, "head dim");
    constexpr int ROWB = 4 * D;            // bytes per key row
    constexpr int QW = ROWB / 16;          // 16-byte words per row
    constexpr int KH = QW > 16 ? 16 : QW;  // words of a key row held at once
    constexpr int NH = QW / KH;            // parts of a key row
    constexpr int DPL = D / 64;            // d per lane in P V
    constexpr int VB = 32;                 // keys of V held at once

    __shared__ __attribute__((aligned(16))) uint4 q_s[RT][QW];
    __shared__ __attribute__((aligned(16))) float p_s[NW][64 * RT];  // [key][row]
    __shared__ __attribute__((aligned(16))) float o_s[NW - 1][RT * D];
    __shared__ float m_s[NW][RT], l_s[NW][RT];
    __shared__ int tab_start[kMaxStreamsPerVideo + 1];
    __shared__ int tab_nlen[kMaxStreamsPerVideo];
    __shared__ int s_total;

    ValuItem it;
    if (!valu_item<RT>(a, it, tab_start, tab_nlen, &s_total)) return;
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const float c = a.qscale;
    const uint32_t stride_b = (uint32_t)a.H_kv * ROWB;

    int row_stream[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) row_stream[r] = r < it.nrows ? (it.row0 + r) / a.G : -2;
    float* const pw = p_s[w];

    // the item's query rows in LDS (rows past nrows are 0)
    for (int i = tid; i < RT * QW; i += 256) {
        const int r = i / QW;
        uint4 x = make_uint4(0u, 0u, 0u, 0u);
        if (r < it.nrows)
            x = reinterpret_cast<const uint4*>(static_cast<const unsigned char*>(a.q) +
                                               (long)row_qrow(a, it.vi, it.id.g, it.row0 + r) * ROWB)[i % QW];
        q_s[r][i % QW] = x;
    }
    __syncthreads();

    float m_ref[RT], l_lane[RT], o[RT][DPL];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        m_ref[r] = -1e30f;
        l_lane[r] = 0.f;
#pragma unroll
        for (int j = 0; j < DPL; ++j) o[r][j] = 0.f;
    }

    for (int u = it.u0 + w; u < it.u1; u += NW) {
        const UnitInfo ui = uniform_unit(unit_info(a, it.vi, it.upre, tab_start, tab_nlen, it.id.g, u));
        const int nk = ui.nk;
        const unsigned char* kb =
            static_cast<const unsigned char*>(ui.stream < 0 ? a.k_prefix : a.k_event) + ui.key_off * 4;
        const unsigned char* vb =
            static_cast<const unsigned char*>(ui.stream < 0 ? a.v_prefix : a.v_event) + ui.key_off * 4;

        // ---- scores, lane = key: the key row in registers, KH words at a time ----
        float sx[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) sx[r] = 0.f;
        const AppendedKey ak = appended_key(a, it.vi, ui, it.id.g, 4);  // fused append: key from k_new / v_new
        const int kk = min(lane, nk - 1);
        const unsigned char* krow = kk == ak.key ? ak.krow : kb + (uint32_t)kk * stride_b;
#pragma unroll
        for (int h = 0; h < NH; ++h) {
            uint4 kx[KH];
#pragma unroll
            for (int j = 0; j < KH; ++j) kx[j] = *reinterpret_cast<const uint4*>(krow + 16 * (h * KH + j));
#pragma unroll
            for (int j = 0; j < KH; ++j) {
                int jj = h * KH + j;
                asm volatile("" : "+s"(jj));
#pragma unroll
                for (int r = 0; r < RT; ++r) {
                    const uint4 q = q_s[r][jj];
                    sx[r] = fmaf(__uint_as_float(q.x), __uint_as_float(kx[j].x), sx[r]);
                    sx[r] = fmaf(__uint_as_float(q.y), __uint_as_float(kx[j].y), sx[r]);
                    sx[r] = fmaf(__uint_as_float(q.z), __uint_as_float(kx[j].z), sx[r]);
                    sx[r] = fmaf(__uint_as_float(q.w), __uint_as_float(kx[j].w), sx[r]);
                }
#pragma unroll
                for (int r = 0; r < RT; ++r) asm volatile("" : "+v"(sx[r]));
            }
        }

        // ---- softmax per row, lane = key ----
        {
            const bool kvalid = lane < nk;
            const bool plan_unit = PLAN && ui.stream < 0 && ui.k0 + kUnit > it.vi.plan0;  // self-only mask
            float pv[RT];
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                bool row_sees = row_stream[r] != -2 && (ui.stream < 0 || row_stream[r] == ui.stream);
                if (plan_unit) row_sees = row_sees & !plan_key_hidden(a, it.vi, ui.k0 + lane, row_stream[r]);
                const float x = (kvalid && row_sees) ? sx[r] * c : kNegInf;
                pv[r] = row_softmax<DPL>(x, m_ref[r], l_lane[r], o[r]);
            }
            float* dst = pw + lane * RT;
            *reinterpret_cast<float4*>(dst) = make_float4(pv[0], pv[1], pv[2], pv[3]);
            *reinterpret_cast<float4*>(dst + 4) = make_float4(pv[4], pv[5], pv[6], pv[7]);
        }
        wave_lds_sync();

        // ---- P V: lane = DPL adjacent d, VB keys of V in flight ----
#pragma unroll
        for (int k0 = 0; k0 < kUnit; k0 += VB) {
            if (k0 >= nk) continue;  // wave-uniform
            float vf[VB][DPL];
#pragma unroll
            for (int k = 0; k < VB; ++k) {
                const int kv = min(k0 + k, nk - 1);
                const float* src =
                    reinterpret_cast<const float*>(kv == ak.key ? ak.vrow : vb + (size_t)kv * stride_b) + lane * DPL;
#pragma unroll
                for (int j = 0; j < DPL; ++j) vf[k][j] = src[j];
            }
#pragma unroll
            for (int k = 0; k < VB; ++k) {
                const float* pr = pw + (k0 + k) * RT;
                const float4 pa = *reinterpret_cast<const float4*>(pr);
                const float4 pb = *reinterpret_cast<const float4*>(pr + 4);
                const float pp[RT] = {pa.x, pa.y, pa.z, pa.w, pb.x, pb.y, pb.z, pb.w};
#pragma unroll
                for (int r = 0; r < RT; ++r)
#pragma unroll
                    for (int j = 0; j < DPL; ++j) o[r][j] = fmaf(pp[r], vf[k][j], o[r][j]);
            }
        }
        wave_lds_sync();  // p_s is rewritten by the next unit
    }

    valu_merge_write<float, D, RT, DPL>(a, it, w, lane, true, lane * DPL, m_ref, l_lane, o, m_s, l_s, o_s[0], o_s[1],
                                 o_s[2]);
}

}  // namespace pdec
