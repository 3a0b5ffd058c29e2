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

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming (non-temporal) 16-byte accesses: the logits and mask rows are
// touched once per step, so they should not evict the classifier table.
__device__ __forceinline__ void store_nt(uint4 *p, uint4 v) {
    u32x4 x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<u32x4 *>(p));
}
__device__ __forceinline__ uint4 load_nt(const uint4 *p) {
    u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(x.x, x.y, x.z, x.w);
}

// Walk of sequence b by one wavefront (Algorithm 2, classification step):
// ref = start[q]; read the stack top-first; stop as soon as ref names a
// class (a determined state).  The walk is a chain of dependent loads, so
// every step is exactly ONE wavefront-wide vector load from the table:
//   sparse row: lane 0 <- (end_class, n_edges), lane 1 <- (default, -),
//               lane j >= 2 <- edge j-2 as (symbol, ref); the edge matching
//               the symbol is found with a ballot and read with readlane;
//   dense row:  lane 0 <- (end_class, -), lane 1 <- entry[symbol];
//   chain:      lane j <- the j-th entry from the current state; lane j
//               compares it with the j-th next stack symbol (a cross-lane
//               shuffle of the staged window), and a ballot finds the first
//               entry the walk does not pass: up to kChunk symbols per load.
// The stack is staged in a window of kChunk symbols in VGPRs (lane j holds
// the j-th symbol below the window's top, stack index chunk_base - j).
// `st` is the stack (len >= 1 symbols, bottom first) and q its lexer state
// (in range).  When the window is restaged, the next row load is issued
// before the window is waited for.  Returns the class id, or -1 for a stack
// symbol out of range; the result is wave-uniform.
constexpr int kChunk = kWave - 1;
static_assert(kSparseMax <= kWave - 2, "a sparse row must fit one wavefront load");
static_assert(kChainMax <= kChunk, "a chain must end within one wavefront load");

constexpr int32_t kRefFault = INT32_MIN;   // no class ref is this small

struct Walk {
    const int32_t *__restrict__ table;
    const int32_t *__restrict__ st;
    int32_t n_lr;
    int lane;
    int i;            // index of the next stack symbol to read (wave-uniform)
    int chunk_base;   // stack index held by window lane 0 (wave-uniform)
    int sym;          // the window (lanes past the bottom hold st[0], never used)
    int ref;          // current state (wave-uniform)
    int cls;          // the result once the walk has ended

    __device__ __forceinline__ void stage() { sym = st[max(chunk_base - lane, 0)]; }

    // One step from a chain entry: lane j holds the j-th entry from the
    // current state.  Returns true when the walk has ended.
    __device__ __forceinline__ bool chain_step(const int4 e) {
        const int pos = chunk_base - i;          // window lane of stack index i
        const int src = pos + lane;              // window lane of stack index i - lane
        const int Xl = __shfl(sym, src & (kWave - 1), kWave);
        const int a = e.x & 0xFFFF;
        const bool pass = a != kSymJump && i - lane >= 0 && src < kChunk && Xl >= 0 && Xl < n_lr &&
                          (a == kSymWild || Xl == a);
        // lane 63 never passes (src >= kChunk), so f <= 63
        const int f = __ffsll((long long)__ballot(!pass)) - 1;
        const int fx = __builtin_amdgcn_readlane(e.x, f);
        if ((fx & 0xFFFF) == kSymJump) {          // end of the chain: go on without reading
            i -= f;
            ref = __builtin_amdgcn_readlane(e.z, f);
            return false;
        }
        if (i - f < 0) { cls = __builtin_amdgcn_readlane(e.w, f); return true; }   // stack ended
        if (pos + f >= kChunk) {                  // window used up: restage, resume at entry f
            i -= f;
            ref = ((ref & ~3) + kChainEntry * f) | kRefChain;
            return false;
        }
        const int fX = __builtin_amdgcn_readlane(Xl, f);
        if (fX < 0 || fX >= n_lr) { cls = -1; return true; }
        i -= f + 1;
        ref = fX == (int)((uint32_t)fx >> 16) ? __builtin_amdgcn_readlane(e.y, f)
                                              : __builtin_amdgcn_readlane(e.z, f);
        return false;
    }

    // One step from a sparse row (lane 0: end_class, n_edges; lane 1:
    // default; lane j >= 2: edge j-2) or a dense row (lane 0: end_class;
    // lane 1: the aligned pair holding entry X).
    __device__ __forceinline__ bool row_step(const int2 v, bool dense, int X) {
        const int va = v.x, vc = v.y;
        if (i < 0) { cls = __builtin_amdgcn_readlane(va, 0); return true; }
        int nref;
        if (dense) {
            nref = (X & 1) ? __builtin_amdgcn_readlane(vc, 1) : __builtin_amdgcn_readlane(va, 1);
        } else {
            const int n = __builtin_amdgcn_readlane(vc, 0);
            const unsigned long long hit = __ballot(lane >= 2 && lane - 2 < n && va == X);
            nref = hit ? __builtin_amdgcn_readlane(vc, __ffsll((long long)hit) - 1)
                       : __builtin_amdgcn_readlane(va, 1);
        }
        // a symbol out of range ends the walk through kRefFault; a select,
        // not a branch, so that the row load cannot sink below the window
        ref = X >= 0 && X < n_lr ? nref : kRefFault;
        i--;
        return false;
    }

    // One step: the one table load, then its evaluation.  A chain or sparse
    // row is loaded before the window is read.
    __device__ __forceinline__ bool step() {
        const int32_t *row = table + (ref & ~3);
        if ((ref & 3) == kRefChain) return chain_step(*reinterpret_cast<const int4 *>(row + kChainEntry * lane));
        if ((ref & 3) == kRefDense) {
            const int X = i >= 0 ? __builtin_amdgcn_readlane(sym, chunk_base - i) : 0;
            const int Xd = X >= 0 && X < n_lr ? X : 0;
            const int2 v = *reinterpret_cast<const int2 *>(row + (lane == 0 ? 0 : kRowHeader + (Xd & ~1)));
            return row_step(v, true, X);
        }
        const int2 v = *reinterpret_cast<const int2 *>(row + 2 * lane);
        const int X = i >= 0 ? __builtin_amdgcn_readlane(sym, chunk_base - i) : 0;
        return row_step(v, false, X);
    }
};

__device__ __forceinline__ int walk_class(const int32_t *__restrict__ table, int32_t n_lr,
                                          const int32_t *__restrict__ st, int len, int q, int lane) {
    Walk w{table, st, n_lr, lane, len - 1, len - 1, 0, 0, -1};
    // round trip 2: the window, with start[q] in lane 63
    w.sym = lane == kChunk ? table[q] : st[max(w.chunk_base - lane, 0)];
    w.ref = __builtin_amdgcn_readlane(w.sym, kChunk);
    if (w.ref < 0) return -w.ref - 1;
    if (w.step()) return w.cls;
    for (;;) {
        // ref, i and chunk_base are wave-uniform; saying so keeps the
        // loop's branches scalar
        w.ref = __builtin_amdgcn_readfirstlane(w.ref);
        w.i = __builtin_amdgcn_readfirstlane(w.i);
        w.chunk_base = __builtin_amdgcn_readfirstlane(w.chunk_base);
        if (w.ref < 0) return w.ref == kRefFault ? -1 : -w.ref - 1;
        if (w.i >= 0 && w.chunk_base - w.i >= kChunk) {
            w.chunk_base = w.i;
            w.stage();
        }
        if (w.step()) return w.cls;
    }
}

// Wavefront 0 of the workgroup walks sequence b; the class (or -1) is
// published to the whole workgroup through LDS.  Slice 0 of each sequence
// counts rejected inputs.  Round trip 1 fetches lens[b], qs[b] and the
// lengths before b (the stack's offset).
__device__ __forceinline__ int block_class(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                           const int32_t *__restrict__ stacks, const int32_t *__restrict__ lens,
                                           const int32_t *__restrict__ qs, int b, uint32_t *__restrict__ err) {
    __shared__ int32_t s_cls;
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        const int own = *((lane & 1) ? qs + b : lens + b);
        int part = lane < b ? lens[lane] : 0;
        for (int i = lane + kWave; i < b; i += kWave) part += lens[i];
        const int len = __builtin_amdgcn_readlane(own, 0);
        const int q = __builtin_amdgcn_readlane(own, 1);
        const int off = wave_sum(part);
        int cls = -1;
        if (len > 0 && q >= 0 && q < n_lex) cls = walk_class(table, n_lr, stacks + off, len, q, lane);
        if (lane == 0) {
            s_cls = cls;
            if (cls < 0 && blockIdx.x == 0) atomicAdd(err, 1u);
        }
    }
    __syncthreads();
    return s_cls;
}

// One workgroup per (sequence b, slice of the mask row): the walk, then the
// whole workgroup copies its slice of the class's precomputed mask row into
// out_bitmask[b] (Algorithm 2, mask step).  Every slice of the same b repeats
// the walk, which costs latency but no HBM bandwidth (the rows are cached).
__global__ void __launch_bounds__(kBlock)
walk_gather_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks,
                   int32_t mask_stride, int32_t n_lex, int32_t n_lr,
                   const int32_t *__restrict__ stacks, const int32_t *__restrict__ lens,
                   const int32_t *__restrict__ qs, int32_t B, int32_t W,
                   uint32_t *__restrict__ out, uint32_t *__restrict__ err, int32_t vec4) {
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int cls = block_class(table, n_lex, n_lr, stacks, lens, qs, b, err);
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
        for (int w = w0 / 4 + tid; w < w1 / 4; w += kBlock) store_nt(d4 + w, load_nt(s4 + w));
    } else {
        for (int w = w0 + tid; w < w1; w += kBlock) dst[w] = src[w];
    }
}

// ---------------------------------------------------------------- apply

constexpr uint16_t kBf16NegInf = 0xFF80u;
constexpr uint32_t kF32NegInf = 0xFF800000u;

// One wavefront applies kWordsPerWave consecutive mask words to the logits
// they cover (the row length V is a multiple of 32 and the logits are 16-byte
// aligned, so word w covers exactly the 32 elements at 32*w).  Lane j holds
// word j in `m` (all ones past the end: nothing to do).  The wavefront writes
// its 64 (bf16) or 32 (fp32) words as kVecs contiguous 1 KiB vector stores;
// lanes get their 8 (bf16) or 4 (fp32) mask bits from the owning lane by a
// cross-lane shuffle.  Entries whose bit is set are never touched: an
// all-zero group is one store of -inf, a mixed group is a read-select-write
// of that 16-byte vector only (all of a lane's reads are issued before its
// stores).
template <bool kBf16>
struct ApplyGeom {
    static constexpr int kPerVec = kBf16 ? 8 : 4;           // elements per 16-byte vector
    static constexpr int kVecsPerWord = 32 / kPerVec;
    static constexpr int kVecs = 4;                         // vectors per lane
    static constexpr int kWordsPerWave = kWave * kVecs / kVecsPerWord;
};

template <bool kBf16>
__device__ __forceinline__ void apply_words(uint4 *__restrict__ base, uint32_t m, int lane) {
    using G = ApplyGeom<kBf16>;
    constexpr uint32_t kFull = (1u << G::kPerVec) - 1;
    uint32_t g[G::kVecs];
    uint4 x[G::kVecs];
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        // vector v = j*64 + lane covers elements [kPerVec*v, kPerVec*v + kPerVec)
        const int v = j * kWave + lane;
        g[j] = (__shfl(m, v / G::kVecsPerWord, kWave) >> ((v % G::kVecsPerWord) * G::kPerVec)) & kFull;
    }
#pragma unroll
    for (int j = 0; j < G::kVecs; j++)
        if (g[j] != 0 && g[j] != kFull) x[j] = load_nt(base + j * kWave + lane);
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        if (g[j] == kFull) continue;
        uint4 val;
        if (g[j] == 0) {
            const uint32_t ni = kBf16 ? (((uint32_t)kBf16NegInf << 16) | kBf16NegInf) : kF32NegInf;
            val = make_uint4(ni, ni, ni, ni);
        } else {
            val = x[j];
            uint32_t *e = reinterpret_cast<uint32_t *>(&val);
            if (kBf16) {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    const uint32_t lo = (g[j] >> (2 * k)) & 1 ? (e[k] & 0xFFFFu) : kBf16NegInf;
                    const uint32_t hi = (g[j] >> (2 * k + 1)) & 1 ? (e[k] >> 16) : kBf16NegInf;
                    e[k] = lo | (hi << 16);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; k++)
                    if (!((g[j] >> k) & 1)) e[k] = kF32NegInf;
            }
        }
        store_nt(base + j * kWave + lane, val);
    }
}

// Fast path of psc_apply_mask: the B rows are one flat run of n_words mask
// words (V % 32 == 0), split over wavefronts.
template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
apply_fast_kernel(uint4 *__restrict__ logits, const uint32_t *__restrict__ bits, int64_t n_words) {
    using G = ApplyGeom<kBf16>;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / kWave) + (threadIdx.x / kWave);
    const int64_t w_base = wave * G::kWordsPerWave;
    if (w_base >= n_words) return;
    uint32_t m = 0xFFFFFFFFu;
    if (lane < G::kWordsPerWave && w_base + lane < n_words) m = bits[w_base + lane];
    apply_words<kBf16>(logits + w_base * G::kVecsPerWord, m, lane);
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

// ---------------------------------------------------------------- fused step

// psc_compute_and_apply, fast path (V % 32 == 0, 16-byte aligned logits):
// one workgroup per (sequence b, slice of kBlock / kWave * kWordsPerWave mask
// words).  After the walk, every wavefront loads its words of the class's
// mask row once, writes them to out_bitmask[b] (when requested) and applies
// them to logits[b] in place.  One launch instead of two, and the bitmask is
// not read back from HBM between the gather and the apply.
template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
fused_fast_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                  int32_t n_lex, int32_t n_lr, const int32_t *__restrict__ stacks,
                  const int32_t *__restrict__ lens, const int32_t *__restrict__ qs, int32_t W,
                  uint32_t *__restrict__ out, uint32_t *__restrict__ err, uint4 *__restrict__ logits) {
    using G = ApplyGeom<kBf16>;
    const int b = blockIdx.y;
    const int cls = block_class(table, n_lex, n_lr, stacks, lens, qs, b, err);
    const int lane = threadIdx.x & (kWave - 1);
    const int w_base = (blockIdx.x * (kBlock / kWave) + threadIdx.x / kWave) * G::kWordsPerWave;
    if (w_base >= W) return;
    uint32_t m = 0xFFFFFFFFu;
    const int w = w_base + lane;
    if (lane < G::kWordsPerWave && w < W) {
        m = cls < 0 ? 0u : masks[(size_t)cls * mask_stride + w];
        if (out) out[(size_t)b * W + w] = m;
    }
    apply_words<kBf16>(logits + ((size_t)b * W + w_base) * G::kVecsPerWord, m, lane);
}

// psc_compute_and_apply, general path (any V, any element alignment): one
// workgroup per (sequence b, kGenWords mask words); the words go through LDS
// and each thread then masks single elements.
constexpr int kGenWords = 128;
static_assert(kGenWords <= kBlock, "one pass stages the slice's words");

template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
fused_generic_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                     int32_t n_lex, int32_t n_lr, const int32_t *__restrict__ stacks,
                     const int32_t *__restrict__ lens, const int32_t *__restrict__ qs, int32_t V, int32_t W,
                     uint32_t *__restrict__ out, uint32_t *__restrict__ err, void *__restrict__ logits) {
    __shared__ uint32_t s_m[kGenWords];
    const int b = blockIdx.y;
    const int cls = block_class(table, n_lex, n_lr, stacks, lens, qs, b, err);
    const int w0 = blockIdx.x * kGenWords;
    const int nw = min(kGenWords, W - w0);
    if (threadIdx.x < nw) {
        const uint32_t m = cls < 0 ? 0u : masks[(size_t)cls * mask_stride + w0 + threadIdx.x];
        s_m[threadIdx.x] = m;
        if (out) out[(size_t)b * W + w0 + threadIdx.x] = m;
    }
    __syncthreads();
    const int e0 = w0 * 32, e1 = min(V, (w0 + nw) * 32);
    for (int e = e0 + threadIdx.x; e < e1; e += kBlock) {
        if ((s_m[(e - e0) >> 5] >> (e & 31)) & 1u) continue;
        const size_t idx = (size_t)b * V + e;
        if (kBf16) reinterpret_cast<uint16_t *>(logits)[idx] = kBf16NegInf;
        else reinterpret_cast<uint32_t *>(logits)[idx] = kF32NegInf;
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
        const int64_t words_per_wave = bf16 ? 64 : 32;           // 4 vectors per lane
        const int64_t waves = (n_words + words_per_wave - 1) / words_per_wave;
        const int64_t blocks = (waves + (kBlock / kWave) - 1) / (kBlock / kWave);
        if (blocks > 0x7FFFFFFF) {
            set_error("psc_apply_mask: tensor too large");
            return PSC_E_INVALID_ARG;
        }
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

extern "C" psc_status psc_compute_and_apply(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                            const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                                            void *logits, psc_dtype dtype, int32_t V, void *stream) {
    if (!h || B < 0 || (dtype != PSC_F32 && dtype != PSC_BF16) ||
        (B > 0 && (!stacks || !stack_lens || !lexer_states || !logits))) {
        set_error("psc_compute_and_apply: null argument, B < 0 or bad dtype");
        return PSC_E_INVALID_ARG;
    }
    if (V != h->V) {
        set_error("psc_compute_and_apply: V (" + std::to_string(V) + ") differs from the vocabulary size (" +
                  std::to_string(h->V) + ")");
        return PSC_E_INVALID_ARG;
    }
    if (!h->dev_base) {
        set_error("psc_compute_and_apply: device tables not bound");
        return PSC_E_NOT_BOUND;
    }
    if (B > 65535) {
        set_error("psc_compute_and_apply: B > 65535");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0) return PSC_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(h->dev_base);
    const int32_t *table = reinterpret_cast<const int32_t *>(base + kTableOff);
    const uint32_t *masks = reinterpret_cast<const uint32_t *>(base + h->mask_off);
    uint32_t *err = reinterpret_cast<uint32_t *>(base);
    const int32_t W = h->W;
    const bool bf16 = dtype == PSC_BF16;
    const bool fast = (V % 32 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
    if (fast) {
        const int words_per_block = (kBlock / kWave) * (bf16 ? ApplyGeom<true>::kWordsPerWave
                                                             : ApplyGeom<false>::kWordsPerWave);
        dim3 grid((W + words_per_block - 1) / words_per_block, B);
        if (bf16)
            hipLaunchKernelGGL(fused_fast_kernel<true>, grid, dim3(kBlock), 0, s, table, masks, h->mask_stride,
                               h->n_lex, h->n_lr, stacks, stack_lens, lexer_states, W, out_bitmask, err,
                               reinterpret_cast<uint4 *>(logits));
        else
            hipLaunchKernelGGL(fused_fast_kernel<false>, grid, dim3(kBlock), 0, s, table, masks, h->mask_stride,
                               h->n_lex, h->n_lr, stacks, stack_lens, lexer_states, W, out_bitmask, err,
                               reinterpret_cast<uint4 *>(logits));
    } else {
        dim3 grid((W + kGenWords - 1) / kGenWords, B);
        if (bf16)
            hipLaunchKernelGGL(fused_generic_kernel<true>, grid, dim3(kBlock), 0, s, table, masks, h->mask_stride,
                               h->n_lex, h->n_lr, stacks, stack_lens, lexer_states, V, W, out_bitmask, err, logits);
        else
            hipLaunchKernelGGL(fused_generic_kernel<false>, grid, dim3(kBlock), 0, s, table, masks,
                               h->mask_stride, h->n_lex, h->n_lr, stacks, stack_lens, lexer_states, V, W,
                               out_bitmask, err, logits);
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail("psc_compute_and_apply", e);
}
