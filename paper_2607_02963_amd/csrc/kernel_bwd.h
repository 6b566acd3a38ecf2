// Backward pass of event-factorized attention over whole branches (the
// training form of the §3.4 mask: query token j of branch e sees every prefix
// token and its own rows 0 .. min(j, n_e - 1)), for one video.
//
// With the forward's O and lse and the incoming dO, for a live query row i
// and a key k it sees:
//   p_ik = 2^(c <q_i, k_k> - lse_i log2 e),  D_i = <dO_i, O_i>,
//   ds_ik = p_ik (<dO_i, v_k> - D_i),
//   dq_i = tau sum_k ds_ik k_k,  dk_k = tau sum_i ds_ik q_i,  dv_k = sum_i p_ik dO_i.
// Rows of ended streams (n_e <= 0) have no output and add nothing.
//
// Three kernels, all on v_mfma_f32_16x16x32_bf16 for the scores and
// v_mfma_f32_16x16x16_bf16 for the products that run over 16 query rows or
// 16 keys:
//  1. D_i for every row (16 lanes per row);
//  2. dk, dv: one work-group per 64-key unit (a prefix unit, or 64 rows of
//     one stream's cache) and kv head; wave w holds keys 16w .. 16w + 15 as
//     the B operands of S = Q K^T and dP = dO V^T, and loops over 64-row
//     tiles of the rows that can see the unit, staged through LDS (four
//     16-row sub-tiles between barriers).  The S
//     accumulator gives a lane key l % 16 for rows 4(l/16) .. +3, which is the
//     A operand (keys x rows) of dV += P^T dO and dK += dS^T Q; their B
//     operands (rows x d) come from the row tiles with the transposing LDS
//     read.  Every key of the unit is written once (0 where no row sees it);
//  3. dq: one work-group per 64 rows and kv head (eight waves: each 16-row
//     block is held by two waves that split each key tile); a wave holds its
//     16 rows as the B operands of S^T = K Q^T and dP^T = V dO^T, and
//     loops over 128-key tiles (prefix, then the own rows of its rows'
//     streams) staged through LDS.  The S^T accumulator gives a lane row
//     l % 16 for keys 4(l/16) .. +3, the A operand (rows x keys) of
//     dQ += dS K, whose B operand (keys x d) is the transposing read of the
//     key tile.
// Tiles are stored with the 16-byte chunks of a row permuted by the row
// index, so the operand reads of 16 rows hit distinct banks.  P and dS meet
// the matrix cores in bf16 (as the forward's P does); every sum is float32.
#pragma once

#include "kernel_mfma.h"

namespace pdec {

constexpr float kLog2eF = 1.44269504088896340736f;

struct BwdArgs {
    const uint16_t* q;     // [E, N, H_q, D]
    const uint16_t* kp;    // [Lmax, H_kv, D]
    const uint16_t* vp;
    const uint16_t* ke;    // [E, cap, H_kv, D]
    const uint16_t* ve;
    const int32_t* event_lens;  // [E]
    const int32_t* prefix_len;  // [1], <= Lmax
    const uint16_t* out;   // [E, N, H_q, D]
    const float* lse;      // [E, N, H_q]
    const uint16_t* dout;  // [E, N, H_q, D]
    float* drow;           // [E * N * H_q]
    float* dq;             // [E, N, H_q, D]
    float* dkp;            // [Lmax, H_kv, D]
    float* dvp;
    float* dke;            // [E, cap, H_kv, D]
    float* dve;
    int E, N, H_q, H_kv, G, cap, Lmax;
    float c;    // tau * log2(e)
    float tau;  // softmax scale
};

__device__ inline f32x4_t mfma_16x16x16(s16x4_t a, s16x4_t b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

__device__ inline s16x4_t pack_bf16x4(float a, float b, float c, float d)
{
    return __builtin_bit_cast(s16x4_t, u32x2_t{pack_bf16x2(a, b), pack_bf16x2(c, d)});
}

// Row r (0 .. E*N*G - 1) of kv head g: stream r / (N G), token (r / G) % N,
// head g G + r % G; its index in q, out, dout, lse and drow.
__device__ inline long bwd_qrow(const BwdArgs& a, int g, int r)
{
    const int e = r / (a.N * a.G), j = (r / a.G) % a.N, hh = r % a.G;
    return ((long)e * a.N + j) * a.H_q + g * a.G + hh;
}

// Byte offset of 16-byte chunk ch of row `row` in a staged tile of D-wide bf16 rows.
template <int D>
__device__ inline int tile_off(int row, int ch)
{
    return row * (2 * D) + 16 * (ch ^ (row % (D / 8)));
}

// Transposing read of a staged tile: lane l receives column 16 dt + l % 16 of
// rows r0 + 4(l/16) .. +3, the B operand (rows x d) of a 16x16x16 product.
template <int D>
__device__ inline s16x4_t tile_tr(const unsigned char* tile, int r0, int dt, int l16, int lg)
{
    const int row = r0 + 4 * lg + (l16 >> 2);
    const int ch = 2 * dt + ((l16 & 3) >> 1);
    const unsigned char* p = tile + tile_off<D>(row, ch) + 8 * (l16 & 1);
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)p);
}

// ---- 1: D_i = <dO_i, O_i> ----
template <int D>
__global__ __launch_bounds__(256) void bwd_drow_kernel(BwdArgs a)
{
    constexpr int PER = D / 16;  // elements per lane, 16 lanes per row
    const long rows = (long)a.E * a.N * a.H_q;
    const long i = (long)blockIdx.x * 16 + threadIdx.x / 16;
    const int l = threadIdx.x % 16;
    float s = 0.f;
    if (i < rows) {
        const uint16_t* o = a.out + i * D + PER * l;
        const uint16_t* d = a.dout + i * D + PER * l;
#pragma unroll
        for (int k = 0; k < PER; ++k)
            s = fmaf(__uint_as_float((uint32_t)o[k] << 16), __uint_as_float((uint32_t)d[k] << 16), s);
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if (i < rows && l == 0) a.drow[i] = s;
}

// ---- 2: dk, dv per 64-key unit ----
template <int D>
__global__ __launch_bounds__(256) void bwd_dkdv_kernel(BwdArgs a)
{
    constexpr int KS = D / 32;  // 32-wide d steps
    constexpr int DT = D / 16;  // 16-wide d blocks
    constexpr int CH = D / 8;   // 16-byte chunks per row
    constexpr int TR = 64;      // rows per staged tile: four 16-row sub-tiles between barriers
    constexpr int SPT = TR * CH / 256;  // staged chunks per thread (q and dO each)
    __shared__ __attribute__((aligned(16))) unsigned char qs[TR * 2 * D];
    __shared__ __attribute__((aligned(16))) unsigned char dos[TR * 2 * D];
    __shared__ float lse2_s[TR], drow_s[TR];
    __shared__ int tok_s[TR];

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, l16 = lane & 15, lg = lane >> 4;
    const int g = blockIdx.y;
    const int UP = (a.Lmax + 63) / 64, UPS = (a.cap + 63) / 64;
    const int u = blockIdx.x;
    const int L = min(max(a.prefix_len[0], 0), a.Lmax);
    const int R = a.E * a.N * a.G;

    // the unit: keys [k0, k0 + 64) of the prefix (own < 0) or of stream own's cache
    int own = -1, k0, kend, nvalid, r_begin, r_end;
    if (u < UP) {
        k0 = 64 * u;
        kend = min(k0 + 64, a.Lmax);
        nvalid = max(0, min(kend, L) - k0);
        r_begin = 0;
        r_end = R;
    } else {
        own = (u - UP) / UPS;
        k0 = 64 * ((u - UP) % UPS);
        kend = min(k0 + 64, a.cap);
        const int nf = a.event_lens[own];
        nvalid = max(0, min(kend, nf) - k0);
        // rows of stream `own` whose token reaches k0
        r_begin = (own * a.N + min(k0, a.N)) * a.G;
        r_end = (own + 1) * a.N * a.G;
        if (nf <= 0) r_end = r_begin;
    }

    // this wave's keys as B operands (zero past the valid ones)
    const int key = k0 + 16 * w + l16;  // the lane's key
    const bool kvalid = key - k0 < nvalid;
    u32x4_t kB[KS], vB[KS];
    {
        const long base = own < 0 ? ((long)key * a.H_kv + g) * D : (((long)own * a.cap + key) * a.H_kv + g) * D;
        const uint16_t* kr = (own < 0 ? a.kp : a.ke) + (kvalid ? base : 0);
        const uint16_t* vr = (own < 0 ? a.vp : a.ve) + (kvalid ? base : 0);
#pragma unroll
        for (int t = 0; t < KS; ++t) {
            kB[t] = kvalid ? *reinterpret_cast<const u32x4_t*>(kr + 32 * t + 8 * lg) : u32x4_t{0u, 0u, 0u, 0u};
            vB[t] = kvalid ? *reinterpret_cast<const u32x4_t*>(vr + 32 * t + 8 * lg) : u32x4_t{0u, 0u, 0u, 0u};
        }
    }
    f32x4_t dk[DT], dv[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        dk[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        dv[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    // row tiles of TR rows, staged through LDS; thread tid moves chunks
    // tid + 256 m of the tile's TR x CH (q and dO) and, for tid < TR, the
    // row's lse, D and token
    auto fetch = [&](int rb, u32x4_t (&qv)[SPT], u32x4_t (&dv4)[SPT], float& l2, float& dr, int& tk) {
#pragma unroll
        for (int m = 0; m < SPT; ++m) {
            const int cidx = tid + 256 * m, sr = cidx / CH, sc = cidx % CH, r = rb + sr;
            qv[m] = dv4[m] = u32x4_t{0u, 0u, 0u, 0u};
            if (r < r_end) {
                const long qr = bwd_qrow(a, g, r);
                qv[m] = *reinterpret_cast<const u32x4_t*>(a.q + qr * D + 8 * sc);
                dv4[m] = *reinterpret_cast<const u32x4_t*>(a.dout + qr * D + 8 * sc);
            }
        }
        l2 = __builtin_inff();  // p = 0 for rows past the range or of ended streams
        dr = 0.f;
        tk = 0;
        if (tid < TR) {
            const int rr = rb + tid;
            if (rr < r_end) {
                const int e = rr / (a.N * a.G);
                const long qr = bwd_qrow(a, g, rr);
                tk = (rr / a.G) % a.N;
                if (a.event_lens[e] > 0) {
                    l2 = a.lse[qr] * kLog2eF;
                    dr = a.drow[qr];
                }
            }
        }
    };

    u32x4_t qv[SPT], dv4[SPT];
    float l2, dr;
    int tk;
    if (r_begin < r_end) fetch(r_begin, qv, dv4, l2, dr, tk);
    for (int rb = r_begin; rb < r_end; rb += TR) {
        __syncthreads();  // the previous tile is no longer read
#pragma unroll
        for (int m = 0; m < SPT; ++m) {
            const int cidx = tid + 256 * m, sr = cidx / CH, sc = cidx % CH;
            *reinterpret_cast<u32x4_t*>(qs + tile_off<D>(sr, sc)) = qv[m];
            *reinterpret_cast<u32x4_t*>(dos + tile_off<D>(sr, sc)) = dv4[m];
        }
        if (tid < TR) {
            lse2_s[tid] = l2;
            drow_s[tid] = dr;
            tok_s[tid] = tk;
        }
        __syncthreads();
        if (rb + TR < r_end) fetch(rb + TR, qv, dv4, l2, dr, tk);  // next tile, in flight meanwhile
        const int nsub = min(TR, r_end - rb + 15) / 16;  // 16-row sub-tiles holding rows of the range

        for (int sub = 0; sub < nsub; ++sub) {
            const int r0 = 16 * sub;
            // S = Q K^T and dP = dO V^T: lane holds rows r0 + 4 lg + i of key l16
            f32x4_t sc4 = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < KS; ++t) {
                const u32x4_t qa = *reinterpret_cast<const u32x4_t*>(qs + tile_off<D>(r0 + l16, 4 * t + lg));
                const u32x4_t da = *reinterpret_cast<const u32x4_t*>(dos + tile_off<D>(r0 + l16, 4 * t + lg));
                sc4 = mfma_16x16x32(as_bf16x8(qa), as_bf16x8(kB[t]), sc4);
                dp = mfma_16x16x32(as_bf16x8(da), as_bf16x8(vB[t]), dp);
            }
            float p[4], ds[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int rr = r0 + 4 * lg + i;
                bool vis = kvalid;
                if (own >= 0) vis = vis & (key <= tok_s[rr]);  // own row t seen by tokens j >= t
                p[i] = vis ? fast_exp2(fmaf(sc4[i], a.c, -lse2_s[rr])) : 0.f;
                ds[i] = p[i] * (dp[i] - drow_s[rr]);
            }
            const s16x4_t pa = pack_bf16x4(p[0], p[1], p[2], p[3]);
            const s16x4_t dsa = pack_bf16x4(ds[0], ds[1], ds[2], ds[3]);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                dv[dt] = mfma_16x16x16(pa, tile_tr<D>(dos, r0, dt, l16, lg), dv[dt]);
                dk[dt] = mfma_16x16x16(dsa, tile_tr<D>(qs, r0, dt, l16, lg), dk[dt]);
            }
        }
    }

    // lane holds keys 16 w + 4 lg + i, d = 16 dt + l16; every key of the unit is written
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int kk = k0 + 16 * w + 4 * lg + i;
        if (kk >= kend) continue;
        const long base = own < 0 ? ((long)kk * a.H_kv + g) * D : (((long)own * a.cap + kk) * a.H_kv + g) * D;
        float* dkr = (own < 0 ? a.dkp : a.dke) + base;
        float* dvr = (own < 0 ? a.dvp : a.dve) + base;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            dkr[16 * dt + l16] = a.tau * dk[dt][i];
            dvr[16 * dt + l16] = dv[dt][i];
        }
    }
}

// ---- 3: dq per 64 rows ----
// Eight waves: wave w takes rows 16 (w % 4) .. +15 of the 64 and half of the
// 16-key blocks of each 128-key tile (the first half for w < 4); the two
// waves of a row block add their dq through LDS at the end.
template <int D>
__global__ __launch_bounds__(512) void bwd_dq_kernel(BwdArgs a)
{
    constexpr int KS = D / 32;
    constexpr int DT = D / 16;
    constexpr int CH = D / 8;
    constexpr int TK = 128;                  // keys per staged tile
    constexpr int PER = TK * CH / 512;       // staged chunks per thread and tile (K or V)
    __shared__ __attribute__((aligned(16))) unsigned char lds[2 * TK * 2 * D];
    unsigned char* ks = lds;                // K tile [TK][D]
    unsigned char* vs = lds + TK * 2 * D;  // V tile [TK][D]

    const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, lg = lane >> 4;
    const int w = (tid >> 6) & 3, kh = tid >> 8;  // row block, key half
    const int g = blockIdx.y;
    const int R = a.E * a.N * a.G;
    const int L = min(max(a.prefix_len[0], 0), a.Lmax);
    const int rw0 = 64 * blockIdx.x;  // first row of the work-group

    // this lane's row (l16 of the wave's 16) as B operands, and its state
    const int row = rw0 + 16 * w + l16;
    const bool rvalid = row < R;
    const int re = rvalid ? row / (a.N * a.G) : 0;
    const int rtok = rvalid ? (row / a.G) % a.N : 0;
    const bool live = rvalid && a.event_lens[re] > 0;
    const long qr = rvalid ? bwd_qrow(a, g, row) : 0;
    const float l2 = live ? a.lse[qr] * kLog2eF : __builtin_inff();
    const float dr = live ? a.drow[qr] : 0.f;
    u32x4_t qB[KS], doB[KS];
#pragma unroll
    for (int t = 0; t < KS; ++t) {
        qB[t] = rvalid ? *reinterpret_cast<const u32x4_t*>(a.q + qr * D + 32 * t + 8 * lg) : u32x4_t{0u, 0u, 0u, 0u};
        doB[t] = rvalid ? *reinterpret_cast<const u32x4_t*>(a.dout + qr * D + 32 * t + 8 * lg)
                        : u32x4_t{0u, 0u, 0u, 0u};
    }
    f32x4_t acc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // key tiles: the prefix, then the cache rows of the streams of this work-group's rows
    const int f_lo = min(rw0, R - 1) / (a.N * a.G), f_hi = min(rw0 + 63, R - 1) / (a.N * a.G);
    const int np = (L + TK - 1) / TK;
    int tiles = np;
    for (int f = f_lo; f <= f_hi; ++f) tiles += (max(a.event_lens[f], 0) + TK - 1) / TK;
    // tile t: (stream or -1, first key, valid keys)
    auto tile_of = [&](int t, int& f, int& t0, int& nv) {
        if (t < np) {
            f = -1;
            t0 = TK * t;
            nv = min(TK, L - t0);
            return;
        }
        t -= np;
        for (f = f_lo; f <= f_hi; ++f) {
            const int nf = max(a.event_lens[f], 0), nt = (nf + TK - 1) / TK;
            if (t < nt) {
                t0 = TK * t;
                nv = min(TK, nf - t0);
                return;
            }
            t -= nt;
        }
        f = -1;
        t0 = 0;
        nv = 0;  // not reached: t < tiles
    };
    // staging: thread tid moves chunks tid + 512 m of the tile's TK x CH (K and V)
    auto fetch = [&](int t, u32x4_t (&kv)[PER], u32x4_t (&vv)[PER]) {
        int f, t0, nv;
        tile_of(t, f, t0, nv);
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int c = tid + 512 * m, kr = c / CH, ch = c % CH;
            kv[m] = vv[m] = u32x4_t{0u, 0u, 0u, 0u};
            if (kr < nv) {
                const long base = f < 0 ? ((long)(t0 + kr) * a.H_kv + g) * D
                                        : (((long)f * a.cap + t0 + kr) * a.H_kv + g) * D;
                kv[m] = *reinterpret_cast<const u32x4_t*>((f < 0 ? a.kp : a.ke) + base + 8 * ch);
                vv[m] = *reinterpret_cast<const u32x4_t*>((f < 0 ? a.vp : a.ve) + base + 8 * ch);
            }
        }
    };

    u32x4_t kv[PER], vv[PER];
    if (tiles > 0) fetch(0, kv, vv);
    for (int t = 0; t < tiles; ++t) {
        int f, t0, nv;
        tile_of(t, f, t0, nv);
        __syncthreads();  // the previous tile is no longer read
#pragma unroll
        for (int m = 0; m < PER; ++m) {
            const int c = tid + 512 * m, kr = c / CH, ch = c % CH;
            *reinterpret_cast<u32x4_t*>(ks + tile_off<D>(kr, ch)) = kv[m];
            *reinterpret_cast<u32x4_t*>(vs + tile_off<D>(kr, ch)) = vv[m];
        }
        __syncthreads();
        if (t + 1 < tiles) fetch(t + 1, kv, vv);  // next tile, in flight meanwhile

#pragma unroll
        for (int kb = (TK / 32) * kh; kb < (TK / 32) * (kh + 1); ++kb) {
            // S^T = K Q^T, dP^T = V dO^T: lane holds keys 16 kb + 4 lg + i of row l16
            f32x4_t s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const u32x4_t ka = *reinterpret_cast<const u32x4_t*>(ks + tile_off<D>(16 * kb + l16, 4 * st + lg));
                const u32x4_t va = *reinterpret_cast<const u32x4_t*>(vs + tile_off<D>(16 * kb + l16, 4 * st + lg));
                s = mfma_16x16x32(as_bf16x8(ka), as_bf16x8(qB[st]), s);
                dp = mfma_16x16x32(as_bf16x8(va), as_bf16x8(doB[st]), dp);
            }
            float ds[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int kk = 16 * kb + 4 * lg + i;  // key within the tile
                bool vis = kk < nv;
                if (f >= 0) vis = vis & (f == re) & (t0 + kk <= rtok);
                const float p = vis ? fast_exp2(fmaf(s[i], a.c, -l2)) : 0.f;
                ds[i] = p * (dp[i] - dr);
            }
            const s16x4_t dsa = pack_bf16x4(ds[0], ds[1], ds[2], ds[3]);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) acc[dt] = mfma_16x16x16(dsa, tile_tr<D>(ks, 16 * kb, dt, l16, lg), acc[dt]);
        }
    }

    // the second key half hands its sums to the first through LDS
    f32x4_t* mbuf = reinterpret_cast<f32x4_t*>(lds);  // [4 row blocks][64 lanes][DT]
    static_assert(4 * 64 * DT * 16 <= 2 * TK * 2 * D, "merge buffer");
    __syncthreads();  // the tiles are no longer read
    if (kh == 1) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) mbuf[(w * 64 + lane) * DT + dt] = acc[dt];
    }
    __syncthreads();
    if (kh == 1) return;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt] += mbuf[(w * 64 + lane) * DT + dt];

    // lane holds rows 16 w + 4 lg + i, d = 16 dt + l16
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = rw0 + 16 * w + 4 * lg + i;
        if (r >= R) continue;
        float* dst = a.dq + bwd_qrow(a, g, r) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) dst[16 * dt + l16] = a.tau * acc[dt][i];
    }
}

}  // namespace pdec
