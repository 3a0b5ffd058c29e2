// psc_probe.hip -- a measurement aid, not part of the mask path: the latency
// of the classifier walk's dependent loads on this GPU, as a function of the
// table's size and of the load's path, in the fused step's launch shape.
//
// The walk of one sequence (Algorithm 2, the classification step) is a chain
// of loads, each address taken from the previous load's data.  This kernel
// makes such a chain through a table of random rows, so the time per extra
// link is the latency of one dependent load under the same launch (grid,
// workgroups of four wavefronts, the walking wavefront's three siblings
// waiting at a barrier and then streaming 4 KiB each of stores, as the step's
// logits stores).

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/psc_probe.h"

namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kRowInts = 256;               // 1 KiB rows
constexpr int32_t kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit elements
constexpr int kPolicyNtDevice = 2 | 16;     // nontemporal, device scope (the step's logits stores)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, kRsrcWord3);
}

// Row index from a loaded value: its magnitude modulo n_rows.
__device__ __forceinline__ int next_row(int v, int n_rows) {
    const int r = v % n_rows;
    return r < 0 ? -r : r;
}

template <int kMode>
__global__ void __launch_bounds__(kBlock)
chase_kernel(uint4 *__restrict__ out, const int32_t *__restrict__ tab, int32_t n_rows, int32_t k, int32_t fill,
             uint32_t seed) {
    __shared__ int32_t s_last;
    const int lane = threadIdx.x & (kWave - 1);
    if (threadIdx.x < kWave) {
        const uint32_t wg = blockIdx.y * gridDim.x + blockIdx.x;
        int x = (int)((wg * 2654435761u + seed * 40503u) % (uint32_t)n_rows);
        for (int i = 0; i < k; i++) {
            const int32_t *row = tab + (size_t)x * kRowInts;
            if (kMode == PSC_PROBE_WAVE_LOAD) {
                // a sparse row's or a chain's load: 16 bytes per lane, 1 KiB per wavefront
                const u32x4 e = __builtin_amdgcn_raw_buffer_load_b128(rsrc(row, kRowInts * 4), lane * 16, 0, 0);
                x = next_row(__builtin_amdgcn_readlane((int)(e[0] ^ e[1] ^ e[2] ^ e[3]), (i * 5) & 63), n_rows);
            } else {
                // a dense row's entry: one uniform address, the scalar path
                x = __builtin_amdgcn_readfirstlane(x);
                const int2 e = *reinterpret_cast<const int2 *>(tab + (size_t)x * kRowInts + 2 * (i & 63));
                x = next_row(e.x ^ e.y, n_rows);
            }
        }
        if (lane == 0) s_last = x;
    }
    __syncthreads();
    if (!fill) return;
    // the step's store stream: four wavefronts, 4 KiB each, one store instruction per 1 KiB
    const int wave = threadIdx.x / kWave;
    const size_t base = ((size_t)(blockIdx.y * gridDim.x + blockIdx.x) * 4 + wave) * 256;
    const u32x4 v = {0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF800000u | (uint32_t)(s_last & 0xFFFF)};
    const __amdgpu_buffer_rsrc_t r = rsrc(out + base, 4096);
#pragma unroll
    for (int j = 0; j < 4; j++) __builtin_amdgcn_raw_buffer_store_b128(v, r, (j * kWave + lane) * 16, 0, kPolicyNtDevice);
}

}  // namespace

extern "C" int psc_probe_chase(int32_t mode, void *out, const int32_t *table, int32_t n_rows, int32_t k,
                               int32_t fill, int32_t grid_x, int32_t grid_y, uint32_t seed, void *stream) {
    if ((mode != PSC_PROBE_WAVE_LOAD && mode != PSC_PROBE_SCALAR_LOAD) || !table || n_rows < 1 || k < 0 ||
        grid_x < 1 || grid_y < 1 || grid_y > 65535 || (int64_t)grid_x * grid_y > (1 << 24) || (fill && !out))
        return (int)hipErrorInvalidValue;
    const dim3 grid((unsigned)grid_x, (unsigned)grid_y);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (mode == PSC_PROBE_WAVE_LOAD)
        hipLaunchKernelGGL(chase_kernel<PSC_PROBE_WAVE_LOAD>, grid, dim3(kBlock), 0, s, static_cast<uint4 *>(out),
                           table, n_rows, k, fill, seed);
    else
        hipLaunchKernelGGL(chase_kernel<PSC_PROBE_SCALAR_LOAD>, grid, dim3(kBlock), 0, s, static_cast<uint4 *>(out),
                           table, n_rows, k, fill, seed);
    return (int)hipGetLastError();
}
