// Matrix-core split pass (bf16, >= 16 query rows per kv head).
//
// The prefix part of the step is a dense contraction: for one kv head, all
// R = E*G query rows of a video against every key of the shared prefix
// (§3.4, Eq. 3).  Each prefix K/V element is read once from HBM and used by
// all R rows.
//
// Work-group = 4 waves; the item's rows (NT tiles of 16) are held by every
// wave, and the item's keys are dealt to the waves in 32-key sub-blocks
// (wave w takes keys [128 b + 32 w, 128 b + 32 w + 32) of block b).  Waves
// never synchronise inside the key loop; at the end their partial states are
// merged through LDS.
//
// Per 32-key sub-block, with v_mfma_f32_16x16x32_bf16 (D = A(16x32) B(32x16)):
//   S^T  = K  Q^T    A = K rows (16 keys x 32 d), B = Q^T (32 d x 16 rows)
//   O^T += V^T P^T   A = V^T (16 d x 32 keys),   B = P^T (32 keys x 16 rows)
// The S^T accumulator gives lane l the scores of query row l%16 for keys
// 4(l/16)..+3 of each 16-key tile, which is exactly a B operand of the second
// product once converted to bf16; so P never leaves registers, and O^T's
// accumulator holds the same query row in the same lane as that row's softmax
// state.  V must have the key as its contraction index: it is written
// transposed into a per-wave LDS tile and read back 8 keys at a time.  For
// both products the k-index order inside a lane only has to agree between A
// and B, which it does by construction.
//
// Softmax: base-2, the q scale folded into the exponent
// (p = 2^(s*c - m)).  The running reference max m is raised only when a tile
// max exceeds it by more than 8 (then O and l are rescaled); otherwise
// p <= 2^8, exact in the final ratio.  Keys past the item are masked to -inf
// and their V rows are zero-filled, never loaded.
#pragma once

#include "pdec_common.h"

namespace pdec {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

__device__ inline f32x4_t mfma_16x16x32(bf16x8_t a, bf16x8_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8_t as_bf16x8(u32x4_t x) { return __builtin_bit_cast(bf16x8_t, x); }

__device__ inline uint32_t pack_bf16x2(float lo, float hi)
{
    const __bf16 a = static_cast<__bf16>(lo), b = static_cast<__bf16>(hi);
    return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int D, int NT>
__global__ __launch_bounds__(256) void split_mfma_kernel(StepArgs a)
{
    constexpr int NW = 4;               // waves per work-group
    constexpr int KSUB = 32;            // keys per wave per block
    constexpr int KBLK = NW * KSUB;     // keys per block
    constexpr int KSTEPS = D / 32;      // k-steps of S^T = K Q^T
    constexpr int DT = D / 16;          // 16-row d tiles of O^T
    constexpr int VCH = KSUB * D / 8 / 64;  // 16-byte V chunks per lane per sub-block
    constexpr int VTS = KSUB + 8;       // LDS row stride (bf16) of the V^T tile
    constexpr int OROW = D + 4;         // LDS row stride (floats) of the merge buffer
    constexpr int LDS_VT = NW * D * VTS * 2;
    constexpr int LDS_MERGE = 2 * NT * 16 * OROW * 4 + 2 * NW * NT * 16 * 4;
    constexpr int LDS_BYTES = LDS_VT > LDS_MERGE ? LDS_VT : LDS_MERGE;
    __shared__ __attribute__((aligned(16))) unsigned char lds[LDS_BYTES];

    Item it;
    if (!decode_item(a, blockIdx.x, it)) return;

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int l16 = lane & 15;  // row (N) / key-in-tile (M) index inside a 16-tile
    const int lg = lane >> 4;   // lane group: selects the k sub-range
    const float c = a.qscale;

    const uint16_t* __restrict__ kp = static_cast<const uint16_t*>(it.prefix ? a.k_prefix : a.k_event) + it.key_off;
    const uint16_t* __restrict__ vp = static_cast<const uint16_t*>(it.prefix ? a.v_prefix : a.v_event) + it.key_off;
    const long stride = (long)a.H_kv * D;

    // Q^T operands: lane holds q[row 16nt + l16][32t + 8lg .. +7], zero for padding rows.
    bf16x8_t qf[NT][KSTEPS];
    {
        const uint16_t* __restrict__ q = static_cast<const uint16_t*>(a.q);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = 16 * nt + l16;
            const bool ok = r < it.nrows;
            const long base = ok ? (long)item_qrow(a, it, r) * D : 0;
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) {
                u32x4_t x = {0u, 0u, 0u, 0u};
                if (ok) x = *reinterpret_cast<const u32x4_t*>(q + base + 32 * t + 8 * lg);
                qf[nt][t] = as_bf16x8(x);
            }
        }
    }

    f32x4_t o[NT][DT];
    float m_ref[NT], l_part[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        m_ref[nt] = kNegInf;
        l_part[nt] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[nt][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    uint16_t* vt = reinterpret_cast<uint16_t*>(lds) + w * D * VTS;
    const int nblocks = (it.nkeys + KBLK - 1) / KBLK;

    u32x4_t kr[2][KSTEPS], vr[VCH];
    auto load_block = [&](int b) {
        const int kb = b * KBLK + w * KSUB;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const int key = kb + 16 * kt + l16;
            const bool ok = key < it.nkeys;
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) {
                u32x4_t x = {0u, 0u, 0u, 0u};
                if (ok) x = *reinterpret_cast<const u32x4_t*>(kp + (long)key * stride + 32 * t + 8 * lg);
                kr[kt][t] = x;
            }
        }
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            const int ch = i * 64 + lane;
            const int key = kb + ch / (D / 8);
            const int d0 = 8 * (ch % (D / 8));
            u32x4_t x = {0u, 0u, 0u, 0u};
            if (key < it.nkeys) x = *reinterpret_cast<const u32x4_t*>(vp + (long)key * stride + d0);
            vr[i] = x;
        }
    };

    if (nblocks > 0) load_block(0);
    for (int b = 0; b < nblocks; ++b) {
        const int kb = b * KBLK + w * KSUB;
        // V^T into this wave's LDS tile; key k = 16 kt + 4 j + i sits at column 8 j + 4 kt + i
#pragma unroll
        for (int i = 0; i < VCH; ++i) {
            const int ch = i * 64 + lane;
            const int k = ch / (D / 8);
            const int d0 = 8 * (ch % (D / 8));
            const int col = 8 * ((k & 15) >> 2) + 4 * (k >> 4) + (k & 3);
            const uint32_t words[4] = {vr[i].x, vr[i].y, vr[i].z, vr[i].w};
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                vt[(d0 + 2 * x) * VTS + col] = (uint16_t)(words[x] & 0xffffu);
                vt[(d0 + 2 * x + 1) * VTS + col] = (uint16_t)(words[x] >> 16);
            }
        }
        bf16x8_t kf[2][KSTEPS];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int t = 0; t < KSTEPS; ++t) kf[kt][t] = as_bf16x8(kr[kt][t]);
        if (b + 1 < nblocks) load_block(b + 1);

        if (kb < it.nkeys) {
            // S^T for the two 16-key tiles and every row tile
            f32x4_t s[2][NT];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int t = 0; t < KSTEPS; ++t) acc = mfma_16x16x32(kf[kt][t], qf[nt][t], acc);
                    s[kt][nt] = acc;
                }
            // mask keys past the item
            if (kb + KSUB > it.nkeys) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (kb + 16 * kt + 4 * lg + i >= it.nkeys) {
#pragma unroll
                            for (int nt = 0; nt < NT; ++nt) s[kt][nt][i] = kNegInf;
                        }
                    }
            }
            // tile max per row (raw score units), shared by the row's 4 lanes
            float mt[NT];
            bool need = false;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                float mx = fmaxf(fmaxf(fmaxf(s[0][nt][0], s[0][nt][1]), fmaxf(s[0][nt][2], s[0][nt][3])),
                                 fmaxf(fmaxf(s[1][nt][0], s[1][nt][1]), fmaxf(s[1][nt][2], s[1][nt][3])));
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                mt[nt] = mx * c;
                need |= mt[nt] > m_ref[nt] + 8.f;
            }
            if (__any(need)) {
                // rows whose own max moved up by more than 8 take the new
                // reference; every other row keeps its reference (alpha = 1,
                // exact), so a row's arithmetic never depends on other rows
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    const bool up = mt[nt] > m_ref[nt] + 8.f;
                    const float mnew = up ? mt[nt] : m_ref[nt];
                    const float alpha = (up && m_ref[nt] != kNegInf) ? fast_exp2(m_ref[nt] - mnew) : 1.f;
                    m_ref[nt] = mnew;
                    l_part[nt] *= alpha;
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) o[nt][dt] *= alpha;
                }
            }
            // P^T operands (bf16) and the normaliser
            bf16x8_t pf[NT];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const float mr = m_ref[nt] == kNegInf ? 0.f : m_ref[nt];
                float p[8];
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) p[4 * kt + i] = fast_exp2(fmaf(s[kt][nt][i], c, -mr));
                float sum = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) sum += p[i];
                l_part[nt] += sum;
                u32x4_t pk = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                              pack_bf16x2(p[6], p[7])};
                pf[nt] = as_bf16x8(pk);
            }
            __builtin_amdgcn_wave_barrier();
            // O^T += V^T P^T
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const u32x4_t vx = *reinterpret_cast<const u32x4_t*>(vt + (16 * dt + l16) * VTS + 8 * lg);
                const bf16x8_t vf = as_bf16x8(vx);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) o[nt][dt] = mfma_16x16x32(vf, pf[nt], o[nt][dt]);
            }
        }
        __builtin_amdgcn_wave_barrier();
    }

    // normaliser: sum the 4 lane groups of each row
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        l_part[nt] += __shfl_xor(l_part[nt], 16);
        l_part[nt] += __shfl_xor(l_part[nt], 32);
    }

    // ---- merge the 4 waves' states through LDS ----
    __syncthreads();  // every wave is done with its V^T tile
    float* obuf0 = reinterpret_cast<float*>(lds);
    float* obuf1 = obuf0 + NT * 16 * OROW;
    float* mbuf = obuf1 + NT * 16 * OROW;  // [NW][NT*16]
    float* lbuf = mbuf + NW * NT * 16;     // [NW][NT*16]
    if (lg == 0) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            mbuf[w * NT * 16 + 16 * nt + l16] = m_ref[nt];
            lbuf[w * NT * 16 + 16 * nt + l16] = l_part[nt];
        }
    }
    __syncthreads();
    float mall[NT], lall[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        float M = kNegInf;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, mbuf[ww * NT * 16 + 16 * nt + l16]);
        float L = 0.f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
            const float mw = mbuf[ww * NT * 16 + 16 * nt + l16];
            L += (mw == kNegInf ? 0.f : fast_exp2(mw - M)) * lbuf[ww * NT * 16 + 16 * nt + l16];
        }
        mall[nt] = M;
        lall[nt] = L;
        const float f = m_ref[nt] == kNegInf ? 0.f : fast_exp2(m_ref[nt] - M);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[nt][dt] *= f;
    }
    auto store_o = [&](float* buf) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                *reinterpret_cast<f32x4_t*>(buf + (16 * nt + l16) * OROW + 16 * dt + 4 * lg) = o[nt][dt];
    };
    auto add_o = [&](const float* buf) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                o[nt][dt] += *reinterpret_cast<const f32x4_t*>(buf + (16 * nt + l16) * OROW + 16 * dt + 4 * lg);
    };
    if (w == 2) store_o(obuf0);
    if (w == 3) store_o(obuf1);
    __syncthreads();
    if (w == 0) add_o(obuf0);
    if (w == 1) add_o(obuf1);
    __syncthreads();
    if (w == 1) store_o(obuf0);
    __syncthreads();
    if (w == 0) {
        add_o(obuf0);
        const long SEH = (long)a.num_events * a.H_q;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int r = 16 * nt + l16;
            if (r < it.nrows) {
                const long qr = item_qrow(a, it, r);
                float* dst = a.part_o + ((long)it.slot * SEH + qr) * D;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<f32x4_t*>(dst + 16 * dt + 4 * lg) = o[nt][dt];
                if (lg == 0) {
                    a.part_m[(long)it.slot * SEH + qr] = mall[nt];
                    a.part_l[(long)it.slot * SEH + qr] = lall[nt];
                }
            }
        }
    }
}

}  // namespace pdec
