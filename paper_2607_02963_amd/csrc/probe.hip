// Read-ceiling probes (measurement aid, pdec_read_probe): how fast the device
// streams a K/V cache pair of the decode step's layout ([L, H_kv, 128] bf16
// each) once, with no arithmetic.  Two access patterns:
//   mode 0  plain reads: each work-group streams a contiguous slab with
//           16-byte loads, eight in flight per thread, the data folded into a
//           checksum word.  The ceiling of a bare read of these bytes in one
//           launch.
//   mode 1  the decode split pass's own memory path: work items (kv head,
//           chunk of keys_per_item keys), every 64-key stage of the head's key
//           and value rows moved by global_load_lds_dwordx4 into a 3-slot LDS
//           ring (two stages in flight), one work-group barrier per stage, as
//           in the split kernels, but nothing computed on the staged keys.
// Nothing is written except the checksum word, and that only when the data
// hash to a fixed value, so the reads cannot be optimised away.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "pdec.h"
#include "pdec_common.h"

namespace {

using namespace pdec;

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
constexpr uint32_t kMagic = 0x9e3779b9u;

__global__ __launch_bounds__(512) void read_plain_kernel(const u32x4_t* k, const u32x4_t* v, long n16, int32_t* sink)
{
    // work-groups 0 .. G/2-1 read K, the others V; each a contiguous slab
    const int half = gridDim.x / 2;
    const bool is_v = (int)blockIdx.x >= half;
    const u32x4_t* src = is_v ? v : k;
    const long per = (n16 + half - 1) / half;
    const long b0 = (long)(is_v ? blockIdx.x - half : blockIdx.x) * per;
    const long b1 = min(n16, b0 + per);
    uint32_t acc = 0;
    for (long i = b0 + threadIdx.x; i < b1; i += 8 * 512) {
        u32x4_t x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const long idx = i + (long)j * 512;
            x[j] = idx < b1 ? src[idx] : u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= x[j].x ^ x[j].y ^ x[j].z ^ x[j].w;
    }
    if (acc == kMagic) sink[0] = (int32_t)acc;
}

__global__ __launch_bounds__(512) void read_ring_kernel(const uint16_t* k, const uint16_t* v, int L, int H, int keys,
                                                        int32_t* sink)
{
    constexpr int NSTAGE = 3, STAGE_K = kUnit * 256, STAGE = 2 * STAGE_K, PIECES = STAGE / 1024, PPW = PIECES / 8;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[NSTAGE * STAGE];
    const int g = blockIdx.x % H, c = blockIdx.x / H;
    const int k0 = c * keys;
    const int nst = (min(L, k0 + keys) - k0 + kUnit - 1) / kUnit;
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // piece p of a stage: keys 4 (p % 16) .. +3 of K (p < 16) or V; lane l
    // moves 16-byte chunk l % 16 of key l / 16 (clamped to the last key)
    auto issue = [&](int st) {
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const int p = w * PPW + i;
            const bool is_v = p >= PIECES / 2;
            const int key = 4 * (p % (PIECES / 2)) + lane / 16;
            const int gk = min(k0 + st * kUnit + key, L - 1);
            const uint16_t* src = (is_v ? v : k) + ((long)gk * H + g) * 128 + 8 * (lane % 16);
            dma_16B(src, lds_u32(lds + (st % NSTAGE) * STAGE + (p % (PIECES / 2)) * 1024 + (is_v ? STAGE_K : 0)));
        }
    };
#pragma unroll
    for (int st = 0; st < NSTAGE - 1; ++st)
        if (st < nst) issue(st);
    uint32_t acc = 0;
    for (int st = 0; st < nst; ++st) {
        if (st + 1 < nst) stage_barrier<PPW>();  // stage st + 1 may be in flight
        else stage_barrier<0>();
        if (st + NSTAGE - 1 < nst) issue(st + NSTAGE - 1);
        acc ^= *reinterpret_cast<const uint32_t*>(lds + (st % NSTAGE) * STAGE + 4 * threadIdx.x);
    }
    if (acc == kMagic) sink[0] = (int32_t)acc;
}

}  // namespace

extern "C" int pdec_read_probe(const void* k, const void* v, int32_t L, int32_t H_kv, int32_t keys_per_item,
                               int32_t mode, int32_t* sink, void* stream)
{
    if (!k || !v || !sink || (reinterpret_cast<uintptr_t>(k) & 15) || (reinterpret_cast<uintptr_t>(v) & 15) ||
        (reinterpret_cast<uintptr_t>(sink) & 3))
        return PDEC_ERR_INVALID_ARG;
    if (L < 1 || H_kv < 1 || (mode != 0 && mode != 1)) return PDEC_ERR_INVALID_ARG;
    if (mode == 1 && (keys_per_item < kUnit || keys_per_item % kUnit != 0)) return PDEC_ERR_INVALID_ARG;
    if ((long)L * H_kv > (1L << 30)) return PDEC_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (mode == 0) {
        const long n16 = (long)L * H_kv * 128 * 2 / 16;
        hipLaunchKernelGGL(read_plain_kernel, dim3(2048), dim3(512), 0, s, static_cast<const u32x4_t*>(k),
                           static_cast<const u32x4_t*>(v), n16, sink);
    } else {
        const long items = (long)H_kv * ((L + keys_per_item - 1) / keys_per_item);
        if (items > INT32_MAX) return PDEC_ERR_UNSUPPORTED;
        hipLaunchKernelGGL(read_ring_kernel, dim3((unsigned)items), dim3(512), 0, s, static_cast<const uint16_t*>(k),
                           static_cast<const uint16_t*>(v), (int)L, (int)H_kv, (int)keys_per_item, sink);
    }
    return hipGetLastError() == hipSuccess ? PDEC_OK : PDEC_ERR_HIP;
}
