// Device side of the mask library (gfx950): table binding, the classifier
// walk + mask gather (Algorithm 2, classification and mask steps), and the
// in-place bitmask -> logits application.
//
// Nothing here is a dense contraction, so no matrix cores are used; the walk
// is a chain of dependent table loads (latency-bound) and the application is
// a pure HBM stream.
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>

#include "psc_internal.hpp"

using namespace psc;

namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;          // 4 wavefronts
constexpr int kCopyWordsPerBlock = 2048;

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// One workgroup per (sequence b, slice of the mask row).  Wavefront 0 walks
// the classifier for sequence b (every slice of the same b repeats the walk,
// which costs latency but no bandwidth), then the whole workgroup copies its
// slice of the class's precomputed mask row into out_bitmask[b].
//
// Walk (Algorithm 2, classification step): ref = start[q]; read the stack
// top-first; each step loads the current row once -- a sparse row as one
// wavefront-wide load of up to 64 (symbol, ref) pairs matched with a ballot,
// a dense row as one indexed load -- and stops as soon as ref names a class
// (a determined state).  The stack is staged 64 symbols at a time in VGPRs
// (lane j holds the j-th symbol from the current top) and read with readlane.
__global__ void __launch_bounds__(kBlock)
walk_gather_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks,
                   int32_t mask_stride, int32_t n_lex, int32_t n_lr,
                   const int32_t *__restrict__ stacks, const int32_t *__restrict__ lens,
                   const int32_t *__restrict__ qs, int32_t B, int32_t W,
                   uint32_t *__restrict__ out, uint32_t *__restrict__ err, int32_t vec4) {
    __shared__ int32_t s_cls;
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    if (tid < kWave) {
        const int lane = tid;
        // start offset of stack b: sum of the lengths before it
        int part = 0;
        for (int i = lane; i < b; i += kWave) part += lens[i];
        const int off = wave_sum(part);
        const int len = lens[b];
        const int q = qs[b];
        int cls = -1;   // -1 = fault
        if (len > 0 && q >= 0 && q < n_lex) {
            const int32_t *st = stacks + off;
            int ref = table[q];
            int i = len - 1;           // index of the next symbol to read
            int chunk_base = i;        // stack index held by lane 0
            int sym = (chunk_base - lane >= 0) ? st[chunk_base - lane] : 0;
            for (;;) {
                if (ref < 0) { cls = -ref - 1; break; }
                const int32_t *row = table + (ref & ~1);
                if (i < 0) { cls = row[0]; break; }
                if (chunk_base - i >= kWave) {
                    chunk_base = i;
                    sym = (chunk_base - lane >= 0) ? st[chunk_base - lane] : 0;
                }
                const int X = __builtin_amdgcn_readlane(sym, chunk_base - i);
                if (X < 0 || X >= n_lr) break;
                if (ref & 1) {
                    ref = row[kRowHeader + X];
                } else {
                    const int n = row[1];
                    const int2 pr = reinterpret_cast<const int2 *>(row + kRowHeader)[lane];
                    const unsigned long long hit = __ballot(lane < n && pr.x == X);
                    ref = hit ? __builtin_amdgcn_readlane(pr.y, __ffsll((long long)hit) - 1) : row[2];
                }
                i--;
            }
        }
        if (lane == 0) {
            s_cls = cls;
            if (cls < 0 && blockIdx.x == 0) atomicAdd(err, 1u);
        }
    }
    __syncthreads();
    const int cls = s_cls;
    const int w0 = blockIdx.x * kCopyWordsPerBlock;
    const int w1 = min(W, w0 + kCopyWordsPerBlock);
    uint32_t *dst = out + (size_t)b * W;
    if (cls < 0) {
        for (int w = w0 + tid; w < w1; w += kBlock) dst[w] = 0u;
        return;
    }
    const uint32_t *src = masks + (size_t)cls * mask_stride;
    if (vec4) {
        // W % 4 == 0 and out is 16-byte aligned: 128-bit loads and stores
        const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
        uint4 *d4 = reinterpret_cast<uint4 *>(dst);
        for (int w = w0 / 4 + tid; w < w1 / 4; w += kBlock) d4[w] = s4[w];
    } else {
        for (int w = w0 + tid; w < w1; w += kBlock) dst[w] = src[w];
    }
}

// ---------------------------------------------------------------- apply

constexpr uint16_t kBf16NegInf = 0xFF80u;
constexpr uint32_t kF32NegInf = 0xFF800000u;

// Fast path: V % 32 == 0 and 16-byte aligned logits, so the flat element
// index is exactly 32 x the flat mask-word index and rows never split a
// vector.  Each wavefront owns 64 consecutive mask words (2048 elements) and
// writes them as contiguous 1 KiB vector stores; lanes get their 8 (bf16) or
// 4 (fp32) mask bits from the owning lane by a cross-lane shuffle.  Entries
// whose bit is set are never touched: an all-zero group is one store of
// -inf, a mixed group is a read-select-write of that 16-byte vector only.
template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
apply_fast_kernel(uint4 *__restrict__ logits, const uint32_t *__restrict__ bits, int64_t n_words) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t seg = (int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave);
    const int64_t w_base = seg * kWave;
    if (w_base >= n_words) return;
    const int64_t wi = w_base + lane;
    const uint32_t m = wi < n_words ? bits[wi] : 0xFFFFFFFFu;
    constexpr int kPerVec = kBf16 ? 8 : 4;          // elements per 16-byte vector
    constexpr int kIters = 32 / kPerVec;            // vectors per mask word
    constexpr uint32_t kFull = (1u << kPerVec) - 1;
    uint4 *base = logits + w_base * kIters;         // 16-byte vectors
#pragma unroll
    for (int j = 0; j < kIters; j++) {
        // vector v = j*64 + lane covers elements [kPerVec*v, kPerVec*v + kPerVec)
        const int v = j * kWave + lane;
        const int src_lane = v / kIters;
        const int shift = (v % kIters) * kPerVec;
        const uint32_t g = (__shfl(m, src_lane, kWave) >> shift) & kFull;
        if (g == kFull) continue;
        if (w_base + src_lane >= n_words) continue;
        uint4 *p = base + v;
        if (g == 0) {
            if (kBf16) {
                const uint32_t ni = ((uint32_t)kBf16NegInf << 16) | kBf16NegInf;
                *p = make_uint4(ni, ni, ni, ni);
            } else {
                *p = make_uint4(kF32NegInf, kF32NegInf, kF32NegInf, kF32NegInf);
            }
        } else {
            uint4 x = *p;
            uint32_t *e = reinterpret_cast<uint32_t *>(&x);
            if (kBf16) {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    uint32_t lo = (g >> (2 * k)) & 1 ? (e[k] & 0xFFFFu) : kBf16NegInf;
                    uint32_t hi = (g >> (2 * k + 1)) & 1 ? (e[k] >> 16) : kBf16NegInf;
                    e[k] = lo | (hi << 16);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; k++)
                    if (!((g >> k) & 1)) e[k] = kF32NegInf;
            }
            *p = x;
        }
    }
}

// General path: any V and alignment, one element per thread.
template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
apply_generic_kernel(void *__restrict__ logits, const uint32_t *__restrict__ bits, int64_t n, int32_t V,
                     int32_t W) {
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += (int64_t)gridDim.x * kBlock) {
        const int64_t b = e / V;
        const int32_t v = (int32_t)(e - b * V);
        if ((bits[b * W + (v >> 5)] >> (v & 31)) & 1u) continue;
        if (kBf16) reinterpret_cast<uint16_t *>(logits)[e] = kBf16NegInf;
        else reinterpret_cast<uint32_t *>(logits)[e] = kF32NegInf;
    }
}

psc_status device_fail(const char *what, hipError_t e) {
    set_error(std::string(what) + ": " + hipGetErrorString(e));
    return PSC_E_DEVICE;
}

}  // namespace

extern "C" psc_status psc_bind_device(psc_handle *h, void *dev_buf, size_t nbytes, void *stream) {
    if (!h || !dev_buf || (reinterpret_cast<uintptr_t>(dev_buf) & 255) != 0) {
        set_error("psc_bind_device: null handle/buffer or buffer not 256-byte aligned");
        return PSC_E_INVALID_ARG;
    }
    size_t need = h->device_bytes_needed();
    if (nbytes < need) {
        set_error("psc_bind_device: buffer too small (" + std::to_string(nbytes) + " < " + std::to_string(need) + ")");
        return PSC_E_INVALID_ARG;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(dev_buf);
    size_t tb = (h->table.size() * sizeof(int32_t) + 255) & ~(size_t)255;
    hipError_t e = hipMemsetAsync(base, 0, kTableOff, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(base + kTableOff, h->table.data(), h->table.size() * sizeof(int32_t),
                           hipMemcpyHostToDevice, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(base + kTableOff + tb, h->masks.data(), h->masks.size() * sizeof(uint32_t),
                           hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return device_fail("psc_bind_device", e);
    h->dev_base = dev_buf;
    h->dev_bytes = nbytes;
    h->mask_off = kTableOff + tb;
    return PSC_OK;
}

extern "C" psc_status psc_compute_masks(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                        const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                                        void *stream) {
    if (!h || B < 0 || (B > 0 && (!stacks || !stack_lens || !lexer_states || !out_bitmask))) {
        set_error("psc_compute_masks: null argument or B < 0");
        return PSC_E_INVALID_ARG;
    }
    if (!h->dev_base) {
        set_error("psc_compute_masks: device tables not bound");
        return PSC_E_NOT_BOUND;
    }
    if (B > 65535) {
        set_error("psc_compute_masks: B > 65535");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0) return PSC_OK;
    char *base = static_cast<char *>(h->dev_base);
    const int32_t W = h->W;
    const int vec4 = (W % 4 == 0) && ((reinterpret_cast<uintptr_t>(out_bitmask) & 15) == 0);
    dim3 grid((W + kCopyWordsPerBlock - 1) / kCopyWordsPerBlock, B);
    hipLaunchKernelGGL(walk_gather_kernel, grid, dim3(kBlock), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const int32_t *>(base + kTableOff),
                       reinterpret_cast<const uint32_t *>(base + h->mask_off), h->mask_stride, h->n_lex, h->n_lr,
                       stacks, stack_lens, lexer_states, B, W, out_bitmask, reinterpret_cast<uint32_t *>(base),
                       vec4);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail("psc_compute_masks", e);
}

extern "C" psc_status psc_apply_mask(void *logits, psc_dtype dtype, const uint32_t *bitmask, int32_t B, int32_t V,
                                     void *stream) {
    if (B < 0 || V < 0 || (dtype != PSC_F32 && dtype != PSC_BF16)) {
        set_error("psc_apply_mask: B/V < 0 or bad dtype");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0 || V == 0) return PSC_OK;
    if (!logits || !bitmask) {
        set_error("psc_apply_mask: null pointer");
        return PSC_E_INVALID_ARG;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool bf16 = dtype == PSC_BF16;
    const int32_t W = (V + 31) / 32;
    const bool fast = (V % 32 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
    if (fast) {
        const int64_t n_words = (int64_t)B * W;
        const int64_t segs = (n_words + kWave - 1) / kWave;
        const int64_t blocks = (segs + (kBlock / kWave) - 1) / (kBlock / kWave);
        if (bf16)
            hipLaunchKernelGGL(apply_fast_kernel<true>, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                               reinterpret_cast<uint4 *>(logits), bitmask, n_words);
        else
            hipLaunchKernelGGL(apply_fast_kernel<false>, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                               reinterpret_cast<uint4 *>(logits), bitmask, n_words);
    } else {
        const int64_t n = (int64_t)B * V;
        const int64_t blocks = std::min<int64_t>((n + kBlock - 1) / kBlock, 65536);
        if (bf16)
            hipLaunchKernelGGL(apply_generic_kernel<true>, dim3((unsigned)blocks), dim3(kBlock), 0, s, logits,
                               bitmask, n, V, W);
        else
            hipLaunchKernelGGL(apply_generic_kernel<false>, dim3((unsigned)blocks), dim3(kBlock), 0, s, logits,
                               bitmask, n, V, W);
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail("psc_apply_mask", e);
}

extern "C" psc_status psc_device_error_count(const psc_handle *h, uint32_t *out, int32_t reset, void *stream) {
    if (!h || !out) {
        set_error("psc_device_error_count: null argument");
        return PSC_E_INVALID_ARG;
    }
    if (!h->dev_base) {
        set_error("psc_device_error_count: device tables not bound");
        return PSC_E_NOT_BOUND;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(out, h->dev_base, sizeof(uint32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && reset) e = hipMemsetAsync(h->dev_base, 0, sizeof(uint32_t), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    return e == hipSuccess ? PSC_OK : device_fail("psc_device_error_count", e);
}
