// Device side of the mask library (gfx950): table binding, the classifier
// walk + mask gather (Algorithm 2, classification and mask steps), the
// in-place bitmask -> logits application, the fused single-launch step (and
// its speculative form and profiling timeline), the masked argmax, and the
// lexing and parsing steps on device-resident prefix states (the advance,
// and the whole decoding step in one launch).  The mask table is read in
// either layout (flat, or deduplicated 64-word slices): kSliced below.
//
// Nothing here is a dense contraction, so no matrix cores are used; the walk
// and the advance are chains of dependent table loads (latency-bound) and
// the application is a pure HBM stream.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "psc_internal.hpp"

using namespace psc;

namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;          // 4 wavefronts
constexpr int kCopyWordsPerBlock = 2048;

// v + v of another lane, moved by a DPP control (kCtrl) into the rows of
// kRowMask (the other rows add zero); 64 bits as two 32-bit moves.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int64_t dpp_add(int64_t v) {
    const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)((uint64_t)v >> 32);
    const uint32_t tlo = (uint32_t)__builtin_amdgcn_update_dpp(0, lo, kCtrl, kRowMask, 0xF, false);
    const uint32_t thi = (uint32_t)__builtin_amdgcn_update_dpp(0, hi, kCtrl, kRowMask, 0xF, false);
    return v + (int64_t)(((uint64_t)thi << 32) | tlo);
}

// The sum of v over the 64 lanes of a full wavefront, uniform.  DPP moves
// instead of LDS-crossbar shuffles: sums of quads (two quad permutes), of
// 8- and 16-lane rows (half-row and row mirrors), then lane 15 of rows 0
// and 2 broadcast into rows 1 and 3, and lane 31 into rows 2 and 3, leaving
// the total in lane 63.
__device__ __forceinline__ int64_t wave_sum(int64_t v) {
    v = dpp_add<0xB1, 0xF>(v);    // quad_perm [1,0,3,2]
    v = dpp_add<0x4E, 0xF>(v);    // quad_perm [2,3,0,1]
    v = dpp_add<0x141, 0xF>(v);   // row_half_mirror
    v = dpp_add<0x140, 0xF>(v);   // row_mirror
    v = dpp_add<0x142, 0xA>(v);   // row_bcast:15
    v = dpp_add<0x143, 0xC>(v);   // row_bcast:31
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), 63);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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

// A raw buffer resource (no stride, no swizzle, 32-bit data format: the
// gfx9-family encoding of the descriptor's last word) over `bytes` bytes at
// p.  Accesses at a byte offset >= bytes are out of range: the hardware
// drops them, and a load returns zeros.
constexpr int32_t kRsrcWord3 = 0x00020000;
constexpr uint32_t kOffSkip = 0x80000000u;   // an offset past any resource used here
constexpr int kPolicyNt = 2;                  // cache policy: nontemporal (streaming)
// Stores of logits: nontemporal at device scope (sc1), so that they are
// written through the XCD's L2 instead of staying dirty in it until the end
// of the kernel (1% faster steps than nontemporal alone on every workload;
// without nontemporal, 13-15% slower).
constexpr int kPolicyStore = kPolicyNt | 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t wave_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, (int32_t)bytes, kRsrcWord3);
}

// Walk of sequence b by one wavefront (Algorithm 2, classification step):
// ref = start[q]; read the stack top-first; stop as soon as ref names a
// class (a determined state).  The walk is a chain of dependent loads, so
// every step is exactly ONE wavefront-wide vector load from the table:
//   sparse row: lane 0 <- (end_class, n_edges), lane 1 <- (default, -),
//               lane j >= 2 <- edge j-2 as (symbol, ref); the edge matching
//               the symbol is found with a ballot and read with readlane;
//   dense row:  entry[symbol] (or the end class) by a scalar load;
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

// With kOverlay, stack indices >= ptr are read from `ov` (the states a
// token pushed, in LDS, not yet written to memory) instead of `st`.
template <bool kOverlay = false, bool kTrack = false>
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
    const int32_t *ov = nullptr;
    int ptr = 0;
    // kTrack: how the last step left its wavefront load -- the lane (sparse
    // row: the matched edge's, or lane 1 for the default; chain: the entry
    // the walk left by) and the kind (0: a sparse edge or a chain entry's
    // second edge; 1: a default or the chain's end); the class predictor's key
    int exit_lane = -1, exit_kind = 0;

    __device__ __forceinline__ int load(int idx) const {
        if (kOverlay && idx >= ptr) return ov[idx - ptr];
        return st[idx];
    }
    __device__ __forceinline__ void stage() { sym = load(max(chunk_base - lane, 0)); }

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
        if (kTrack) {
            exit_lane = f;
            exit_kind = 1;
        }
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
        if (kTrack) exit_kind = fX == (int)((uint32_t)fx >> 16) ? 0 : 1;
        ref = fX == (int)((uint32_t)fx >> 16) ? __builtin_amdgcn_readlane(e.y, f)
                                              : __builtin_amdgcn_readlane(e.z, f);
        return false;
    }

    // One step from a sparse row, 16 bytes per lane: lane 0 (end_class,
    // n_edges), lane 1 (-, default, default's skip), lane j >= 2 edge j - 2
    // (symbol, ref, skip); the edge matching the symbol is found with a
    // ballot and read with readlane.  A skip of k wildcard entries then reads
    // the next k symbols from the window without a load (only their range is
    // checked) and goes on at the chain's jump target, as the chain would;
    // when the stack ends within them, they reach past the window, or one is
    // out of range, the walk takes the chain itself.
    __device__ __forceinline__ bool row_step(const int4 v, int X) {
        if (i < 0) { cls = __builtin_amdgcn_readlane(v.x, 0); return true; }
        const int n = __builtin_amdgcn_readlane(v.y, 0);
        const unsigned long long hit = __ballot(lane >= 2 && lane - 2 < n && v.x == X);
        const int h = hit ? __ffsll((long long)hit) - 1 : 1;
        const int nref = __builtin_amdgcn_readlane(v.y, h);
        const int nskip = __builtin_amdgcn_readlane(v.z, h);
        if (kTrack) {
            exit_lane = h;
            exit_kind = 0;
        }
        // a symbol out of range ends the walk through kRefFault; a select,
        // not a branch, so that the row load cannot sink below the window
        const bool ok = X >= 0 && X < n_lr;
        ref = ok ? nref : kRefFault;
        i--;
        if (ok) take_skip(nskip);
        return false;
    }

    // After a row step: read the k wildcard symbols of `skip` from the window
    // and go on at its target, when they are all there and in range.
    __device__ __forceinline__ void take_skip(int skip) {
        if (skip == kNoSkip) return;
        const int k = (int)((uint32_t)skip >> 27);
        const int lo = chunk_base - i;          // window lane of stack index i
        const unsigned long long valid = __ballot(sym >= 0 && sym < n_lr);
        if (i - (k - 1) >= 0 && lo + k <= kChunk) {
            const unsigned long long need = ((1ull << k) - 1) << lo;
            if ((valid & need) == need) {
                i -= k;
                ref = (int)(((uint32_t)skip & ((1u << 27) - 1)) - (1u << 26));
            }
        }
    }

    // The first step from start[q], whose wavefront load (the start block)
    // was fetched together with the window; a dense row still reads its entry.
    __device__ __forceinline__ bool first_step(const int4 blk) {
        if ((ref & 3) == kRefChain) return chain_step(blk);
        if ((ref & 3) == kRefDense) return step();
        const int X = i >= 0 ? __builtin_amdgcn_readlane(sym, chunk_base - i) : 0;
        return row_step(blk, X);
    }

    // One step: the one table load, then its evaluation.  A chain or sparse
    // row is loaded before the window is read.
    __device__ __forceinline__ bool step() {
        const int32_t *row = table + (ref & ~3);
        if ((ref & 3) == kRefChain) return chain_step(*reinterpret_cast<const int4 *>(row + kChainEntry * lane));
        if ((ref & 3) == kRefDense) {
            // one uniform address: a scalar load of the entry (ref, skip)
            if (i < 0) { cls = row[0]; return true; }
            const int X = __builtin_amdgcn_readlane(sym, chunk_base - i);
            const bool ok = X >= 0 && X < n_lr;
            const int2 e = *reinterpret_cast<const int2 *>(row + kRowHeader + 2 * (ok ? X : 0));
            ref = ok ? e.x : kRefFault;
            i--;
            if (ok) take_skip(e.y);
            return false;
        }
        const int4 v = *reinterpret_cast<const int4 *>(row + kSparseEdge * lane);
        const int X = i >= 0 ? __builtin_amdgcn_readlane(sym, chunk_base - i) : 0;
        return row_step(v, X);
    }
};

// The start blocks sit just below the table: block q (kStartBlockInts int32)
// starts (nb - q) blocks before it, nb = start_block_count(n_lex) (n_lex >= 1
// here: q is in range).  A higher q loads block nb - 1 in its place and
// takes its first step as any other.
template <bool kOverlay = false>
__device__ __forceinline__ int walk_class(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                          const int32_t *__restrict__ st, int len, int q, int lane,
                                          const int32_t *ov = nullptr, int ptr = 0) {
    Walk<kOverlay> w{table, st, n_lr, lane, len - 1, len - 1, 0, 0, -1, ov, ptr};
    // round trip 2: the window, with start[q] in lane 63, and start[q]'s
    // first wavefront load from the start block
    const int nb = start_block_count(n_lex);
    u32x4 bv = reinterpret_cast<const u32x4 *>(table - (int64_t)(nb - min(q, nb - 1)) * kStartBlockInts)[lane];
    w.sym = lane == kChunk ? table[q] : w.load(max(w.chunk_base - lane, 0));
    // both loads are needed here, as whole registers: this keeps the compiler
    // from sinking the block's load below the wait for the window, or waiting
    // for it before the window's load is issued
    asm volatile("" : "+v"(bv), "+v"(w.sym));
    w.ref = __builtin_amdgcn_readlane(w.sym, kChunk);
    if (w.ref < 0) return -w.ref - 1;
    if (q >= nb) {
        // no start block: the same load from the row itself
        const int32_t *row = table + (w.ref & ~3);
        if ((w.ref & 3) != kRefDense) bv = *reinterpret_cast<const u32x4 *>(row + 4 * lane);
    }
    if (w.first_step(make_int4((int)bv[0], (int)bv[1], (int)bv[2], (int)bv[3]))) return w.cls;
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

// A walk in two parts, for the class predictor (Walk with kTrack): begin()
// makes round trip 2 (the window, start[q] and its start block, and q's
// predictor entries) and the first step; finish() walks on to the class.
// After begin(), `done` says whether the class is already known (in `cls`);
// otherwise `slot` is the predictor entry that the way the first step left
// the start block keys (-1: none) and `pc` the class recorded there (-1:
// none).  The predictor entries of q are int32 [64 lanes][2 kinds].
struct WalkRun {
    Walk<false, true> w;
    bool done;
    int cls, slot, pc;

    __device__ __forceinline__ void begin(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                          int32_t n_classes, const int32_t *__restrict__ st, int len, int q,
                                          int lane, const int32_t *__restrict__ pred) {
        w = Walk<false, true>{table, st, n_lr, lane, len - 1, len - 1, 0, 0, -1, nullptr, 0};
        done = false;
        cls = -1;
        slot = -1;
        pc = -1;
        const int nb = start_block_count(n_lex);
        const int qb = min(q, nb - 1);
        u32x4 bv = reinterpret_cast<const u32x4 *>(table - (int64_t)(nb - qb) * kStartBlockInts)[lane];
        u32x2 pv = reinterpret_cast<const u32x2 *>(pred + (int64_t)qb * kPredInts)[lane];
        w.sym = lane == kChunk ? table[q] : w.load(max(w.chunk_base - lane, 0));
        asm volatile("" : "+v"(bv), "+v"(pv), "+v"(w.sym));
        w.ref = __builtin_amdgcn_readlane(w.sym, kChunk);
        if (w.ref < 0) {
            done = true;
            cls = -w.ref - 1;
            return;
        }
        const bool has_block = q < nb;
        if (!has_block) {
            const int32_t *row = table + (w.ref & ~3);
            if ((w.ref & 3) != kRefDense) bv = *reinterpret_cast<const u32x4 *>(row + 4 * lane);
        }
        const bool dense = (w.ref & 3) == kRefDense;
        if (w.first_step(make_int4((int)bv[0], (int)bv[1], (int)bv[2], (int)bv[3]))) {
            done = true;
            cls = w.cls;
            return;
        }
        if (has_block && !dense) {
            slot = (qb * kWave + w.exit_lane) * 2 + w.exit_kind;
            const int p = __builtin_amdgcn_readlane((int)(w.exit_kind ? pv[1] : pv[0]), w.exit_lane);
            pc = p >= 0 && p < n_classes ? p : -1;
        }
    }

    __device__ __forceinline__ int finish() {
        for (;;) {
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
};

// The lengths of sequences i0 + k * kWave + lane, k < kN, loaded in one
// round trip (every load issued before the first is used), negative ones as
// zero, summed per lane.
constexpr int kLensPerRound = 4;

template <int kN>
__device__ __forceinline__ int64_t lens_round(__amdgpu_buffer_rsrc_t rl, int i0, int lane) {
    int v[kN];
#pragma unroll
    for (int k = 0; k < kN; k++)
        v[k] = (int)__builtin_amdgcn_raw_buffer_load_b32(rl, (uint32_t)(i0 + k * kWave + lane) * 4u, 0, 0);
    int64_t sum = 0;
#pragma unroll
    for (int k = 0; k < kN; k++) sum += max(v[k], 0);
    return sum;
}

// One wavefront walks sequence b and returns its class, or -1 for an input
// out of range.  Round trip 1 fetches lens[b], qs[b] and, for ragged stacks
// (stride 0), the lengths before b (more round trips past 64 sequences):
// the stack's offset, summed in 64 bits
// (the stacks may hold more than 2^31 symbols in all), a negative length
// counting as zero; a ragged stack reaching past n_stack symbols is an input
// out of range, never read.  With stride > 0 stack b starts at b * stride
// and holds at most stride symbols.
__device__ __forceinline__ int wave_class(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                          const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack,
                                          const int32_t *__restrict__ lens, const int32_t *__restrict__ qs,
                                          int b, int lane) {
    const int own = *((lane & 1) ? qs + b : lens + b);
    int64_t part = 0;
    if (stride == 0) {
        // a buffer resource over lens[0..b) turns the loads past b into
        // zeros without a branch
        const __amdgpu_buffer_rsrc_t rl = wave_rsrc(lens, (uint32_t)b * 4u);
        if (b <= kWave) {
            part = lens_round<1>(rl, 0, lane);
        } else {
            for (int i0 = 0; i0 < b; i0 += kLensPerRound * kWave) part += lens_round<kLensPerRound>(rl, i0, lane);
        }
    }
    const int len = __builtin_amdgcn_readlane(own, 0);
    const int q = __builtin_amdgcn_readlane(own, 1);
    const int64_t off = stride ? (int64_t)b * stride : wave_sum(part);
    if (len > 0 && (stride == 0 ? off + len <= n_stack : len <= stride) && q >= 0 && q < n_lex)
        return walk_class(table, n_lex, n_lr, stacks + off, len, q, lane);
    return -1;
}

// Wavefront 0 of the workgroup walks sequence b; the class (or -1) is
// published to the whole workgroup through LDS.  Slice 0 of each sequence
// counts rejected inputs.
__device__ __forceinline__ int block_class(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                           const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack,
                                           const int32_t *__restrict__ lens, const int32_t *__restrict__ qs,
                                           int b, uint32_t *__restrict__ err) {
    __shared__ int32_t s_cls;
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        const int cls = wave_class(table, n_lex, n_lr, stacks, stride, n_stack, lens, qs, b, lane);
        if (lane == 0) {
            s_cls = cls;
            if (cls < 0 && blockIdx.x == 0) atomicAdd(err, 1u);
        }
    }
    __syncthreads();
    return s_cls;
}

// Round trip 1 and the start of the tracked walk of sequence b (the
// predictor's form of wave_class): r.done with class -1 for an input out of
// range.
__device__ __forceinline__ void wave_begin(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr,
                                           int32_t n_classes, const int32_t *__restrict__ stacks, int32_t stride,
                                           int64_t n_stack, const int32_t *__restrict__ lens,
                                           const int32_t *__restrict__ qs, const int32_t *__restrict__ pred, int b,
                                           int lane, WalkRun &r) {
    const int own = *((lane & 1) ? qs + b : lens + b);
    int64_t part = 0;
    if (stride == 0) {
        const __amdgpu_buffer_rsrc_t rl = wave_rsrc(lens, (uint32_t)b * 4u);
        if (b <= kWave) {
            part = lens_round<1>(rl, 0, lane);
        } else {
            for (int i0 = 0; i0 < b; i0 += kLensPerRound * kWave) part += lens_round<kLensPerRound>(rl, i0, lane);
        }
    }
    const int len = __builtin_amdgcn_readlane(own, 0);
    const int q = __builtin_amdgcn_readlane(own, 1);
    const int64_t off = stride ? (int64_t)b * stride : wave_sum(part);
    if (len > 0 && (stride == 0 ? off + len <= n_stack : len <= stride) && q >= 0 && q < n_lex) {
        r.begin(table, n_lex, n_lr, n_classes, stacks + off, len, q, lane, pred);
    } else {
        r.done = true;
        r.cls = -1;
        r.slot = -1;
        r.pc = -1;
    }
}

// After a tracked walk: record its class in the predictor entry its first
// step keyed, when it differs from the prediction, and count the update.
// Lane 0 of one wavefront per sequence.
__device__ __forceinline__ void pred_update(int32_t *__restrict__ pred, uint32_t *__restrict__ counters,
                                            const WalkRun &r, int cls) {
    if (!r.done && r.slot >= 0 && cls >= 0 && cls != r.pc) {
        pred[r.slot] = cls;
        atomicAdd(counters + kCounterPredUpdates, 1u);
    }
}

// psc_compute_classes: the walk alone (Algorithm 2, classification step),
// one wavefront per sequence, kBlock / kWave sequences per workgroup.  It
// fills the class predictor that the speculative step reads.
__global__ void __launch_bounds__(kBlock)
classes_kernel(const int32_t *__restrict__ table, int32_t n_lex, int32_t n_lr, int32_t n_classes,
               const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack, const int32_t *__restrict__ lens,
               const int32_t *__restrict__ qs, int32_t B, int32_t *__restrict__ out, uint32_t *__restrict__ counters,
               int32_t *__restrict__ pred) {
    const int b = blockIdx.x * (kBlock / kWave) + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (b >= B) return;
    const int lane = threadIdx.x & (kWave - 1);
    WalkRun r;
    wave_begin(table, n_lex, n_lr, n_classes, stacks, stride, n_stack, lens, qs, pred, b, lane, r);
    const int cls = r.done ? r.cls : r.finish();
    if (lane == 0) {
        out[b] = cls;
        if (cls < 0) atomicAdd(counters + kCounterFaults, 1u);
        pred_update(pred, counters, r, cls);
    }
}

// Word w of class c's mask row: rows[c * stride + w] in the flat layout;
// with kSliced, rows[ids[c * stride + w / 64] * 64 + w % 64] (each distinct
// 64-word slice of the rows stored once; stride = slices per row).
template <bool kSliced>
__device__ __forceinline__ const uint32_t *mask_at(const uint32_t *__restrict__ rows, int32_t stride,
                                                   const int32_t *__restrict__ ids, int c, int w) {
    if (kSliced)
        return rows + (int64_t)ids[(int64_t)c * stride + (w >> 6)] * kSliceWords + (w & (kSliceWords - 1));
    return rows + (int64_t)c * stride + w;
}

// One workgroup per (sequence b, slice of the mask row): the walk, then the
// whole workgroup copies its slice of the class's precomputed mask row into
// out_bitmask[b] (Algorithm 2, mask step).  Every slice of the same b repeats
// the walk, which costs latency but no HBM bandwidth (the rows are cached).
template <bool kSliced>
__global__ void __launch_bounds__(kBlock)
walk_gather_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks,
                   int32_t mask_stride, const int32_t *__restrict__ ids, int32_t n_lex, int32_t n_lr,
                   const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack,
                   const int32_t *__restrict__ lens, const int32_t *__restrict__ qs, int32_t B, int32_t W,
                   uint32_t *__restrict__ out, uint32_t *__restrict__ err, int32_t vec4) {
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int cls = block_class(table, n_lex, n_lr, stacks, stride, n_stack, lens, qs, b, err);
    const int w0 = blockIdx.x * kCopyWordsPerBlock;
    const int w1 = min(W, w0 + kCopyWordsPerBlock);
    uint32_t *dst = out + (size_t)b * W;
    if (cls < 0) {
        for (int w = w0 + tid; w < w1; w += kBlock) dst[w] = 0u;
        return;
    }
    const uint32_t *src = masks + (size_t)cls * mask_stride;   // the flat layout's row
    if (vec4) {
        // W % 4 == 0 and out is 16-byte aligned: 128-bit loads and stores
        // every load is issued before the first store, so no store waits
        // for another to complete
        const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
        uint4 *d4 = reinterpret_cast<uint4 *>(dst);
        constexpr int kPer = kCopyWordsPerBlock / 4 / kBlock;
        uint4 v[kPer];
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int w = w0 / 4 + tid + k * kBlock;
            if (w < w1 / 4)
                v[k] = kSliced ? load_nt(reinterpret_cast<const uint4 *>(mask_at<true>(masks, mask_stride, ids, cls, 4 * w)))
                               : load_nt(s4 + w);
        }
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int w = w0 / 4 + tid + k * kBlock;
            if (w < w1 / 4) store_nt(d4 + w, v[k]);
        }
    } else {
        for (int w = w0 + tid; w < w1; w += kBlock) dst[w] = *mask_at<kSliced>(masks, mask_stride, ids, cls, w);
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

//
// The loads and stores go through a buffer resource over the wavefront's
// `bytes` bytes of logits.  A lane that must not touch its vector gets an
// offset past the end instead of a branch: the hardware drops such an access
// (a load returns zeros) without a memory request.  Every memory instruction
// is then issued unconditionally, so the compiler counts them exactly: the
// selects wait for their loads only, and no store waits for an earlier
// store to complete (with branches it had to wait for all outstanding
// accesses before each vector, which serialised the stores).
template <bool kBf16>
__device__ __forceinline__ void apply_words(uint4 *__restrict__ base, uint32_t bytes, uint32_t m, int lane) {
    using G = ApplyGeom<kBf16>;
    constexpr uint32_t kFull = (1u << G::kPerVec) - 1;
    const __amdgpu_buffer_rsrc_t rsrc = wave_rsrc(base, bytes);
    uint32_t g[G::kVecs];
    u32x4 x[G::kVecs];
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        // vector v = j*64 + lane covers elements [kPerVec*v, kPerVec*v + kPerVec)
        const int v = j * kWave + lane;
        g[j] = (__shfl(m, v / G::kVecsPerWord, kWave) >> ((v % G::kVecsPerWord) * G::kPerVec)) & kFull;
    }
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        const uint32_t off = (uint32_t)(j * kWave + lane) * 16u;
        x[j] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, g[j] != 0 && g[j] != kFull ? off : kOffSkip, 0,
                                                     kPolicyNt);
    }
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        u32x4 val = x[j];
        if (kBf16) {
#pragma unroll
            for (int k = 0; k < 4; k++) {
                const uint32_t lo = (g[j] >> (2 * k)) & 1 ? (val[k] & 0xFFFFu) : kBf16NegInf;
                const uint32_t hi = (g[j] >> (2 * k + 1)) & 1 ? (val[k] >> 16) : kBf16NegInf;
                val[k] = lo | (hi << 16);
            }
        } else {
#pragma unroll
            for (int k = 0; k < 4; k++)
                if (!((g[j] >> k) & 1)) val[k] = kF32NegInf;
        }
        const uint32_t off = (uint32_t)(j * kWave + lane) * 16u;
        __builtin_amdgcn_raw_buffer_store_b128(val, rsrc, g[j] != kFull ? off : kOffSkip, 0, kPolicyStore);
    }
}

// Fast path of psc_apply_mask: the B rows are one flat run of n_words mask
// words (V % 32 == 0), split over wavefronts.
template <bool kBf16>
__global__ void __launch_bounds__(kBlock)
apply_fast_kernel(uint4 *__restrict__ logits, const uint32_t *__restrict__ bits, int64_t n_words) {
    using G = ApplyGeom<kBf16>;
    const int lane = threadIdx.x & (kWave - 1);
    // the wavefront index is uniform: saying so keeps the buffer resource in
    // scalar registers
    const int64_t wave = (int64_t)blockIdx.x * (kBlock / kWave) +
                         __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t w_base = wave * G::kWordsPerWave;
    if (w_base >= n_words) return;
    uint32_t m = 0xFFFFFFFFu;
    if (lane < G::kWordsPerWave && w_base + lane < n_words) m = bits[w_base + lane];
    const uint32_t words = (uint32_t)min<int64_t>(G::kWordsPerWave, n_words - w_base);
    apply_words<kBf16>(logits + w_base * G::kVecsPerWord, words * G::kVecsPerWord * 16u, m, lane);
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
// one workgroup per (sequence b, slice of kFusedBlock / kWave *
// kWordsPerWave mask words).  After the walk, every wavefront loads its words
// of the class's mask row once, writes them to out_bitmask[b] (when
// requested) and applies them to logits[b] in place.  One launch instead of
// two, and the bitmask is not read back from HBM between the gather and the
// apply.  Four wavefronts per workgroup (2 measured slightly faster on a
// 200-step schema sample but slower over the 1,000-step schema workload and
// on the largest one); the walk is repeated per workgroup, which costs
// latency but no bandwidth.
constexpr int kFusedBlock = 4 * kWave;

// The part of the fused step after the walk: this workgroup's slice of the
// class's mask row, written to out_bitmask[b] and applied to logits[b].
template <bool kBf16, bool kSliced>
__device__ __forceinline__ void fused_fast_apply(int cls, int b, const uint32_t *__restrict__ masks,
                                                 int32_t mask_stride, const int32_t *__restrict__ ids, int32_t W,
                                                 uint32_t *__restrict__ out, uint4 *__restrict__ logits) {
    using G = ApplyGeom<kBf16>;
    const int lane = threadIdx.x & (kWave - 1);
    const int w_base =
        (blockIdx.x * (kFusedBlock / kWave) + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave)) * G::kWordsPerWave;
    if (w_base >= W) return;
    uint32_t m = 0xFFFFFFFFu;
    const int w = w_base + lane;
    const bool mine = lane < G::kWordsPerWave && w < W;
    if (mine) m = cls < 0 ? 0u : *mask_at<kSliced>(masks, mask_stride, ids, cls, w);
    const uint32_t words = (uint32_t)min(G::kWordsPerWave, W - w_base);
    apply_words<kBf16>(logits + ((size_t)b * W + w_base) * G::kVecsPerWord, words * G::kVecsPerWord * 16u, m,
                       lane);
    // last, so that the logits accesses never wait for this store
    if (out && mine) out[(size_t)b * W + w] = m;
}

// A timeline record per wavefront (psc_compute_and_apply_timeline): its
// start, the prediction known (t_a), its class known (t_b) and its last
// store issued, in ticks of the GPU's constant 100 MHz clock; then the
// wavefront, its XCD, whether the prediction held and whether the class was
// known at the first step; then the sequence and the slice.
__device__ __forceinline__ void timeline_record(unsigned long long *__restrict__ tl, unsigned long long t0,
                                                unsigned long long t_a, unsigned long long t_b, uint32_t held,
                                                uint32_t early) {
    const unsigned long long t_e = wall_clock64();
    const uint32_t wave = threadIdx.x / kWave;
    const uint32_t xcc = __builtin_amdgcn_s_getreg((20) | (0 << 6) | (3 << 11)) & 15u;   // XCC_ID[3:0]
    const size_t rec = ((size_t)blockIdx.y * gridDim.x + blockIdx.x) * (blockDim.x / kWave) + wave;
    unsigned long long *o = tl + rec * 4;
    o[0] = t0;
    o[1] = (t_a - t0) | ((t_b - t0) << 32);
    o[2] = (t_e - t0) | ((unsigned long long)(wave | (xcc << 3) | (held << 7) | (early << 8)) << 32);
    o[3] = (unsigned long long)blockIdx.y | ((unsigned long long)blockIdx.x << 32);
}

// kTl: the timeline variant (profiling records, psc_compute_and_apply_timeline).
template <bool kBf16, bool kSliced, bool kTl>
__global__ void __launch_bounds__(kFusedBlock)
fused_fast_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                  const int32_t *__restrict__ ids, int32_t n_lex, int32_t n_lr, const int32_t *__restrict__ stacks,
                  int32_t stride, int64_t n_stack, const int32_t *__restrict__ lens, const int32_t *__restrict__ qs,
                  int32_t W, uint32_t *__restrict__ out, uint32_t *__restrict__ err, uint4 *__restrict__ logits,
                  unsigned long long *__restrict__ tl) {
    unsigned long long t0 = 0, t_b = 0;
    if (kTl) t0 = wall_clock64();
    const int b = blockIdx.y;
    const int cls = block_class(table, n_lex, n_lr, stacks, stride, n_stack, lens, qs, b, err);
    if (kTl) t_b = wall_clock64();
    fused_fast_apply<kBf16, kSliced>(cls, b, masks, mask_stride, ids, W, out, logits);
    if (kTl && (threadIdx.x & (kWave - 1)) == 0) timeline_record(tl, t0, t0, t_b, 0u, 0u);
}

// psc_compute_and_apply, general path (any V, any element alignment): one
// workgroup per (sequence b, kGenWords mask words); the words go through LDS
// and each thread then masks single elements.
constexpr int kGenWords = 128;
static_assert(kGenWords <= kBlock, "one pass stages the slice's words");

template <bool kBf16, bool kSliced>
__device__ __forceinline__ void fused_generic_apply(int cls, int b, const uint32_t *__restrict__ masks,
                                                    int32_t mask_stride, const int32_t *__restrict__ ids, int32_t V,
                                                    int32_t W, uint32_t *__restrict__ out,
                                                    void *__restrict__ logits) {
    __shared__ uint32_t s_m[kGenWords];
    const int w0 = blockIdx.x * kGenWords;
    const int nw = min(kGenWords, W - w0);
    if (threadIdx.x < nw) {
        const uint32_t m = cls < 0 ? 0u : *mask_at<kSliced>(masks, mask_stride, ids, cls, w0 + threadIdx.x);
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

template <bool kBf16, bool kSliced>
__global__ void __launch_bounds__(kBlock)
fused_generic_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                     const int32_t *__restrict__ ids, int32_t n_lex, int32_t n_lr, const int32_t *__restrict__ stacks,
                     int32_t stride, int64_t n_stack, const int32_t *__restrict__ lens,
                     const int32_t *__restrict__ qs, int32_t V, int32_t W, uint32_t *__restrict__ out,
                     uint32_t *__restrict__ err, void *__restrict__ logits) {
    const int b = blockIdx.y;
    const int cls = block_class(table, n_lex, n_lr, stacks, stride, n_stack, lens, qs, b, err);
    fused_generic_apply<kBf16, kSliced>(cls, b, masks, mask_stride, ids, V, W, out, logits);
}

// The speculative form of psc_compute_and_apply's fast path
// (PSC_OPT_SPECULATE).  Wavefront 0 walks with the class predictor: after its
// first step (two round trips in) it publishes the predicted class, or the
// class itself when the walk has already ended (barrier A).  Wavefronts 1-3
// then load their mask words of that class, and the logits vectors those
// words leave partly allowed (the only ones whose old values the in-place
// select needs), while the walk goes on; at barrier B, when the walk ends in
// that class, they select and store at once, and otherwise load that
// class's words and the partly allowed vectors they do not hold yet.
// Wavefront 0 applies its own words after the walk, as in fused_fast_kernel.
// Every result is that of fused_fast_kernel.
struct SpecShared {
    int32_t pc, done, cls;
};

template <bool kBf16>
__device__ __forceinline__ void vector_groups(uint32_t m, int lane, uint32_t (&g)[ApplyGeom<kBf16>::kVecs]) {
    using G = ApplyGeom<kBf16>;
    constexpr uint32_t kFull = (1u << G::kPerVec) - 1;
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        const int v = j * kWave + lane;
        g[j] = (__shfl(m, v / G::kVecsPerWord, kWave) >> ((v % G::kVecsPerWord) * G::kPerVec)) & kFull;
    }
}

template <bool kBf16>
__device__ __forceinline__ bool mixed_group(uint32_t g) {
    constexpr uint32_t kFull = (1u << ApplyGeom<kBf16>::kPerVec) - 1;
    return g != 0 && g != kFull;
}

template <bool kBf16, bool kSliced, bool kTl>
__global__ void __launch_bounds__(kFusedBlock)
fused_spec_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                  const int32_t *__restrict__ ids, int32_t n_lex, int32_t n_lr, int32_t n_classes,
                  const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack,
                  const int32_t *__restrict__ lens, const int32_t *__restrict__ qs, int32_t W,
                  uint32_t *__restrict__ out, uint32_t *__restrict__ counters, int32_t *__restrict__ pred,
                  uint4 *__restrict__ logits, unsigned long long *__restrict__ tl) {
    using G = ApplyGeom<kBf16>;
    constexpr uint32_t kFull = (1u << G::kPerVec) - 1;
    __shared__ SpecShared sh;
    unsigned long long t0 = 0, t_a = 0, t_b = 0;
    if (kTl) t0 = wall_clock64();
    const int b = blockIdx.y;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x & (kWave - 1);
    WalkRun r;
    if (wave == 0) {
        wave_begin(table, n_lex, n_lr, n_classes, stacks, stride, n_stack, lens, qs, pred, b, lane, r);
        if (lane == 0) {
            sh.done = r.done;
            sh.pc = r.done ? r.cls : r.pc;
        }
    }
    __syncthreads();                                             // A
    if (kTl) t_a = wall_clock64();
    const int done = sh.done, pc = sh.pc;
    const int w_base = (blockIdx.x * (kFusedBlock / kWave) + wave) * G::kWordsPerWave;
    const bool active = w_base < W;
    const int w = w_base + lane;
    const bool mine = active && lane < G::kWordsPerWave && w < W;
    const uint32_t words = active ? (uint32_t)min(G::kWordsPerWave, W - w_base) : 0u;
    const __amdgpu_buffer_rsrc_t rsrc =
        wave_rsrc(logits + ((size_t)b * W + (active ? w_base : 0)) * G::kVecsPerWord, words * G::kVecsPerWord * 16u);
    const bool have = wave > 0 && (done || pc >= 0);
    uint32_t mp = 0xFFFFFFFFu, gp[G::kVecs];
    u32x4 xp[G::kVecs];
#pragma unroll
    for (int j = 0; j < G::kVecs; j++) {
        gp[j] = kFull;
        xp[j] = u32x4{0u, 0u, 0u, 0u};
    }
    int cls = -1;
    if (wave == 0) {
        cls = r.done ? r.cls : r.finish();
        if (lane == 0) sh.cls = cls;
    } else if (have && active) {
        if (mine) mp = pc < 0 ? 0u : *mask_at<kSliced>(masks, mask_stride, ids, pc, w);
        vector_groups<kBf16>(mp, lane, gp);
#pragma unroll
        for (int j = 0; j < G::kVecs; j++) {
            const uint32_t off = (uint32_t)(j * kWave + lane) * 16u;
            xp[j] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, mixed_group<kBf16>(gp[j]) ? off : kOffSkip, 0,
                                                          kPolicyNt);
        }
    }
    if (!done) __syncthreads();                                  // B
    if (kTl) t_b = wall_clock64();
    cls = done ? pc : sh.cls;
    if (active) {
        uint32_t m = mp, g[G::kVecs];
        u32x4 x[G::kVecs];
#pragma unroll
        for (int j = 0; j < G::kVecs; j++) {
            g[j] = gp[j];
            x[j] = xp[j];
        }
        if (!(have && cls == pc)) {
            m = 0xFFFFFFFFu;
            if (mine) m = cls < 0 ? 0u : *mask_at<kSliced>(masks, mask_stride, ids, cls, w);
            vector_groups<kBf16>(m, lane, g);
            u32x4 y[G::kVecs];
#pragma unroll
            for (int j = 0; j < G::kVecs; j++) {
                const uint32_t off = (uint32_t)(j * kWave + lane) * 16u;
                const bool need = mixed_group<kBf16>(g[j]) && !mixed_group<kBf16>(gp[j]);
                y[j] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, need ? off : kOffSkip, 0, kPolicyNt);
            }
#pragma unroll
            for (int j = 0; j < G::kVecs; j++)
                if (!mixed_group<kBf16>(gp[j])) x[j] = y[j];
        }
#pragma unroll
        for (int j = 0; j < G::kVecs; j++) {
            u32x4 val = x[j];
            if (kBf16) {
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    const uint32_t lo = (g[j] >> (2 * k)) & 1 ? (val[k] & 0xFFFFu) : kBf16NegInf;
                    const uint32_t hi = (g[j] >> (2 * k + 1)) & 1 ? (val[k] >> 16) : kBf16NegInf;
                    val[k] = lo | (hi << 16);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; k++)
                    if (!((g[j] >> k) & 1)) val[k] = kF32NegInf;
            }
            const uint32_t off = (uint32_t)(j * kWave + lane) * 16u;
            __builtin_amdgcn_raw_buffer_store_b128(val, rsrc, g[j] != kFull ? off : kOffSkip, 0, kPolicyStore);
        }
        // last, so that the logits accesses never wait for this store
        if (out && mine) out[(size_t)b * W + w] = m;
    }
    if (wave == 0 && lane == 0 && blockIdx.x == 0) {
        if (cls < 0) atomicAdd(counters + kCounterFaults, 1u);
        pred_update(pred, counters, r, cls);
    }
    if (kTl && lane == 0) timeline_record(tl, t0, t_a, t_b, (uint32_t)(!done && cls == pc), (uint32_t)done);
}

// ---------------------------------------------------------------- masked argmax

// Greedy decoding folded into the mask step: out[b] = the allowed token with
// the largest logit (ties to the lowest id; NaN above everything; -1 if no
// token is allowed).  The logits are only read, and only the 16-byte vectors
// holding at least one allowed token.  One launch with the fused step's
// workgroups (one per sequence and slice of the row): each folds its best
// (value, id) key into the sequence's slot with a 64-bit atomic max, then
// counts itself in the sequence's arrival counter; the workgroup that
// arrives last takes the slot (an atomic exchange with zero), clears the
// counter and writes the token.  Slot and counter are touched only by
// device-scope atomics, which every XCD performs at the same point, and a
// workgroup's counter increment is issued only after its max has returned,
// so the last arrival sees every max without a fence (a device-scope release
// would write back a whole L2 on this GPU).  Both are zero between calls.
// Each sequence's slot and counter share a 128-byte record of their own:
// with 32 counters packed in a cache line, the atomics queued on that line
// cost 1.5 us per C3 step.

// An order-preserving key: larger float, larger key; NaN above +inf; -0 = +0.
__device__ __forceinline__ uint32_t order_key(uint32_t u) {
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0xFFFFFFFFu;
    if (u == 0x80000000u) u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ unsigned long long arg_key(uint32_t fbits, int v) {
    return ((unsigned long long)order_key(fbits) << 32) | (0xFFFFFFFFu - (uint32_t)v);
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
    return a > b ? a : b;
}

template <bool kBf16, bool kSliced>
__global__ void __launch_bounds__(kFusedBlock)
argmax_partial_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                      const int32_t *__restrict__ ids, int32_t n_lex, int32_t n_lr,
                      const int32_t *__restrict__ stacks, int32_t stride, int64_t n_stack,
                      const int32_t *__restrict__ lens, const int32_t *__restrict__ qs, int32_t V, int32_t W,
                      uint32_t *__restrict__ err, const void *__restrict__ logits, int32_t fast,
                      unsigned long long *__restrict__ records, int32_t *__restrict__ out_tokens) {
    using G = ApplyGeom<kBf16>;
    __shared__ unsigned long long s_best[kFusedBlock / kWave];
    const int b = blockIdx.y;
    const int cls = block_class(table, n_lex, n_lr, stacks, stride, n_stack, lens, qs, b, err);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    unsigned long long best = 0;   // every real key is > 0
    if (cls >= 0) {
        if (fast) {
            // the apply's layout: the wavefront's kWordsPerWave words, lane j
            // the vectors j, j + 64, ...; only vectors with an allowed token are read
            constexpr uint32_t kFull = (1u << G::kPerVec) - 1;
            const int w0 = (blockIdx.x * (kFusedBlock / kWave) + wave) * G::kWordsPerWave;
            if (w0 < W) {
                const uint4 *row = reinterpret_cast<const uint4 *>(logits) + ((size_t)b * W + w0) * G::kVecsPerWord;
                const uint32_t m =
                    lane < G::kWordsPerWave && w0 + lane < W ? *mask_at<kSliced>(masks, mask_stride, ids, cls, w0 + lane)
                                                             : 0u;
                uint32_t g[G::kVecs];
                uint4 x[G::kVecs];
#pragma unroll
                for (int j = 0; j < G::kVecs; j++) {
                    const int v = j * kWave + lane;
                    g[j] = (__shfl(m, v / G::kVecsPerWord, kWave) >> ((v % G::kVecsPerWord) * G::kPerVec)) & kFull;
                }
#pragma unroll
                for (int j = 0; j < G::kVecs; j++)
                    if (g[j]) x[j] = load_nt(row + j * kWave + lane);
#pragma unroll
                for (int j = 0; j < G::kVecs; j++) {
                    if (!g[j]) continue;
                    const uint32_t *e = reinterpret_cast<const uint32_t *>(&x[j]);
                    const int v0 = (w0 * G::kVecsPerWord + j * kWave + lane) * G::kPerVec;
#pragma unroll
                    for (int k = 0; k < G::kPerVec; k++) {
                        if (!((g[j] >> k) & 1)) continue;
                        const uint32_t f = kBf16 ? ((k & 1) ? (e[k / 2] & 0xFFFF0000u) : (e[k / 2] << 16)) : e[k];
                        best = umax64(best, arg_key(f, v0 + k));
                    }
                }
            }
        } else {
            const int v_end = min(V, (blockIdx.x + 1) * kGenWords * 32);
            for (int v = blockIdx.x * kGenWords * 32 + threadIdx.x; v < v_end; v += kFusedBlock) {
                if (!((*mask_at<kSliced>(masks, mask_stride, ids, cls, v >> 5) >> (v & 31)) & 1u)) continue;
                const size_t idx = (size_t)b * V + v;
                const uint32_t f = kBf16 ? (uint32_t)reinterpret_cast<const uint16_t *>(logits)[idx] << 16
                                         : reinterpret_cast<const uint32_t *>(logits)[idx];
                best = umax64(best, arg_key(f, v));
            }
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) best = umax64(best, __shfl_xor(best, o, kWave));
    if (lane == 0) s_best[wave] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int k = 1; k < kFusedBlock / kWave; k++) best = umax64(best, s_best[k]);
        unsigned long long *slot = records + (size_t)b * kArgmaxRecordWords;
        uint32_t *arrivals = reinterpret_cast<uint32_t *>(slot + 1);
        const unsigned long long seen = __hip_atomic_fetch_max(slot, best, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        // the max has been performed once its old value is back
        asm volatile("s_waitcnt vmcnt(0)" ::"v"((uint32_t)seen) : "memory");
        const uint32_t arrived = __hip_atomic_fetch_add(arrivals, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (arrived == gridDim.x - 1) {
            const unsigned long long k = __hip_atomic_exchange(slot, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_exchange(arrivals, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            out_tokens[b] = k ? (int32_t)(0xFFFFFFFFu - (uint32_t)k) : -1;
        }
    }
}

// ---------------------------------------------------------------- allocation-free argmax records

// The argmax slot records of psc_compute_and_argmax_noalloc: a fixed array
// in the library's own device memory, one copy per GPU, held until the
// process ends (kScratchSeqs records of 128 bytes: 512 KiB).  Host code
// never uses this name as an address (it is a host-side stand-in there):
// it uses the per-device address that hipGetSymbolAddress returns.
constexpr int32_t kScratchSeqs = 4096;
static __device__ __align__(256) unsigned long long scratch[kScratchSeqs * kArgmaxRecordWords];

// Zero n uint64 words (the records' state between calls), with vector stores.
__global__ void __launch_bounds__(kBlock)
zero_words_kernel(unsigned long long *__restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) p[i] = 0;
}

// ---------------------------------------------------------------- advance

// The problem instance on the device (the lexing and parsing steps of
// Algorithm 2, which turn a prefix state and a token into the next state).
struct AdvTables {
    const int32_t *lex_next, *lex_accept, *ignored, *action, *go, *prod_lhs, *prod_len, *tok_off;
    const uint8_t *bytes;
    int32_t n_lex, n_lr, n_term, n_nt, end_term, eos, V;
    int32_t packed;    // action holds packed reductions (kind | len << 2 | lhs << 10)
    const int32_t *closure;   // GOTO with the following unit reductions done, or null
};

constexpr int kOverlay = 192;          // states one token may push above what it keeps
// Bound on the LR steps that feeding one terminal may take.  A parse of any
// stack ends long before it: every reduction that does not shrink the stack
// is a unit or an empty one, at most one per nonterminal before the stack
// shrinks or grows (an LR grammar has no derivation cycles), and growth
// stops at the capacity.  The bound only keeps a wave from spinning on
// tables or stacks that are not what they should be.
__device__ __forceinline__ int64_t feed_step_bound(int32_t n_nt, int len, int cap) {
    return (int64_t)(n_nt + 2) * (4 * (int64_t)len + 4 * (int64_t)cap + 8) + 65536;
}

// One wavefront advances one sequence by one token.  Everything it computes
// is uniform across the wavefront (the sequence is the workgroup's), so the
// table reads are scalar loads with one address each, and no sequence waits
// for another's path through the lexer and the parser.  The token's bytes
// are fetched up front, 64 at a time, one per lane.  While the token is
// processed the kept part of the stack, stacks[b][0 .. ptr), is only read
// and the states pushed above it live in an LDS overlay, so a rejected token
// leaves the stack, its length and the lexer state exactly as they were; on
// success the overlay is written above ptr.  A terminal is fed as the LR
// parser does: the reductions its lookahead selects, then a shift (accept
// for $end); popping the whole stack or a missing goto rejects.
//
// advance_core computes the outcome of token `tok` on the state (q_in, st
// of `len` symbols, at most `cap`) and writes nothing but the overlay: on
// PSC_ADV_OK the new state is st[0 .. ptr) followed by s_ov[0 .. ov), in
// lexer state q; on any other status the state is unchanged (ptr = len,
// ov = 0, q = q_in).
__device__ __forceinline__ int advance_core(const AdvTables &T, int32_t *s_ov, const int32_t *__restrict__ st,
                                            int len, int q_in, int tok, int cap, int lane, int &ptr_out,
                                            int &ov_out, int &q_out) {
    ptr_out = len;
    ov_out = 0;
    q_out = q_in;
    if (tok < 0) return PSC_ADV_SKIPPED;
    if (tok >= T.V || len < 1 || len > cap || q_in < 0 || q_in >= T.n_lex) return PSC_ADV_BAD_INPUT;
    int ptr = len, ov = 0;
    int32_t cur = st[ptr - 1];   // the top of the stack, kept in a register
    auto reload = [&]() { cur = __builtin_amdgcn_readfirstlane(ov > 0 ? s_ov[ov - 1] : st[ptr - 1]); };
    auto push = [&](int32_t x) {
        if (ov >= kOverlay) return false;
        s_ov[ov++] = x;          // every lane writes the same value
        cur = x;
        return true;
    };
    // states come from the tables (validated when built) or, below the
    // overlay, from the caller's stack, which is checked before each use
    const int64_t max_steps = feed_step_bound(T.n_nt, len, cap);
    auto feed = [&](int32_t t) -> int {
        for (int64_t guard = 0; guard < max_steps; guard++) {
            const int32_t s0 = cur;
            if (s0 < 0 || s0 >= T.n_lr) return PSC_ADV_BAD_INPUT;
            const int32_t a = T.action[(int64_t)s0 * T.n_term + t];
            const int kind = a & 3;
            if (kind == 1) return push(a >> 2) ? PSC_ADV_OK : PSC_ADV_OVERFLOW;
            if (kind == 3) return PSC_ADV_OK;
            if (kind == 0) return PSC_ADV_REJECTED;
            int32_t lhs;
            int k;
            if (T.packed) {
                lhs = a >> 10;
                k = (a >> 2) & 255;
            } else {
                const int32_t p = a >> 2;
                lhs = T.prod_lhs[p];
                k = T.prod_len[p];
            }
            const int from_ov = min(k, ov);
            ov -= from_ov;
            k -= from_ov;
            if (k >= ptr) return PSC_ADV_REJECTED;       // nothing left to goto from
            ptr -= k;
            reload();
            const int32_t s1 = cur;
            if (s1 < 0 || s1 >= T.n_lr) return PSC_ADV_BAD_INPUT;
            // with the closure, the unit reductions the lookahead selects
            // next are done here too (each would pop the state just pushed
            // and push a GOTO from s1): the stack ends the same
            const int32_t g = T.closure ? T.closure[((int64_t)s1 * T.n_nt + lhs) * T.n_term + t]
                                        : T.go[(int64_t)s1 * T.n_nt + lhs];
            if (g < 0) return PSC_ADV_REJECTED;
            if (!push(g)) return PSC_ADV_OVERFLOW;
        }
        return PSC_ADV_REJECTED;
    };
    int q = q_in, res = PSC_ADV_OK;
    if (tok == T.eos) {
        // the pending lexeme becomes its terminal, then $end must be accepted
        res = PSC_ADV_EOS;
        if (q != 0) {
            const int32_t t = T.lex_accept[q];
            if (t < 0) res = PSC_ADV_REJECTED;
            else if (!T.ignored[t]) {
                const int r = feed(t);
                if (r != PSC_ADV_OK) res = r;
            }
        }
        if (res == PSC_ADV_EOS) {
            const int r = feed(T.end_term);
            if (r != PSC_ADV_OK) res = r;
        }
        return res;
    }
    // longest match with one byte of lookahead: a byte the pending lexeme
    // cannot take ends it (it must be accepting) and starts the next from q0
    const int i0 = T.tok_off[tok], n = T.tok_off[tok + 1] - i0;
    for (int base = 0; base < n && res == PSC_ADV_OK; base += kWave) {
        const int chunk = __builtin_amdgcn_readfirstlane(min(kWave, n - base));
        const int byte = lane < chunk ? T.bytes[i0 + base + lane] : 0;
        for (int j = 0; j < chunk; j++) {
            const int c = __builtin_amdgcn_readlane(byte, j);
            const int32_t nx = T.lex_next[(int64_t)q * 256 + c];
            if (nx >= 0) { q = nx; continue; }
            const int32_t t = q != 0 ? T.lex_accept[q] : -1;
            if (t < 0) { res = PSC_ADV_REJECTED; break; }
            if (!T.ignored[t]) {
                res = feed(t);
                if (res != PSC_ADV_OK) break;
            }
            q = T.lex_next[c];
            if (q < 0) { res = PSC_ADV_REJECTED; break; }
        }
    }
    if (res == PSC_ADV_OK && ptr + ov > cap) res = PSC_ADV_OVERFLOW;
    if (res == PSC_ADV_OK) {
        ptr_out = ptr;
        ov_out = ov;
        q_out = q;
    }
    return res;
}

// psc_advance: one workgroup of one wavefront per sequence, the state
// updated in place.
__global__ void __launch_bounds__(kWave)
advance_kernel(AdvTables T, int32_t *__restrict__ stacks, int32_t cap, int32_t *__restrict__ lens,
               int32_t *__restrict__ qs, int32_t B, const int32_t *__restrict__ tokens,
               int32_t *__restrict__ status) {
    __shared__ int32_t s_ov[kOverlay];
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int tok = tokens[b];
    const int len = tok < 0 ? 0 : lens[b], q_in = tok < 0 ? 0 : qs[b];
    int ptr, ov, q;
    const int res = advance_core(T, s_ov, stacks + (int64_t)b * cap, len, q_in, tok, cap, lane, ptr, ov, q);
    if (res == PSC_ADV_OK) {
        int32_t *dst = stacks + (int64_t)b * cap + ptr;
        for (int k = lane; k < ov; k += kWave) dst[k] = s_ov[k];
        if (lane == 0) {
            lens[b] = ptr + ov;
            qs[b] = q;
        }
    }
    if (lane == 0) status[b] = res;
}

// Every sequence back to the empty prefix: lexer state q0, stack [0].
__global__ void __launch_bounds__(kBlock)
reset_kernel(int32_t *__restrict__ stacks, int32_t cap, int32_t *__restrict__ lens, int32_t *__restrict__ qs,
             int32_t B) {
    const int b = blockIdx.x * kBlock + threadIdx.x;
    if (b >= B) return;
    stacks[(int64_t)b * cap] = 0;
    lens[b] = 1;
    qs[b] = 0;
}

// ---------------------------------------------------------------- decoding step

// The state a decoding step reads and the one it writes (dense layout,
// separate buffers: every workgroup of a sequence reads the old state while
// the first one writes the new state).
struct DecodeArgs {
    AdvTables T;
    const int32_t *stacks_in, *lens_in, *qs_in;
    int32_t *stacks_out, *lens_out, *qs_out;
    const int32_t *tokens;
    int32_t *status;
    int32_t cap;
};

// Algorithm 2 for sequence b in one workgroup: wavefront 0 advances the
// prefix state by tokens[b] (advance_core: the pushed states stay in the LDS
// overlay), walks the new state (the kept part of the stack from memory,
// the pushed states from the overlay) and publishes the class; the
// sequence's first workgroup also writes the new state and the status.  A
// token that is not advanced leaves the state as it was, and that state is
// the one classified, exactly as psc_advance followed by
// psc_compute_and_apply_dense.
__device__ __forceinline__ int decode_block_class(const int32_t *__restrict__ table, const DecodeArgs &D, int b,
                                                  uint32_t *__restrict__ err) {
    __shared__ int32_t s_cls;
    __shared__ int32_t s_ov[kOverlay];
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        const int cap = D.cap;
        const int tok = D.tokens[b];
        const int len = D.lens_in[b], q_in = D.qs_in[b];
        const int32_t *st = D.stacks_in + (int64_t)b * cap;
        int ptr, ov, q;
        const int res = advance_core(D.T, s_ov, st, len, q_in, tok, cap, lane, ptr, ov, q);
        const int new_len = res == PSC_ADV_OK ? ptr + ov : len;
        if (blockIdx.x == 0) {
            int32_t *dst = D.stacks_out + (int64_t)b * cap;
            const int keep = res == PSC_ADV_OK ? ptr : min(max(len, 0), cap);
            for (int k = lane; k < keep; k += kWave) dst[k] = st[k];
            for (int k = lane; k < ov; k += kWave) dst[ptr + k] = s_ov[k];
            if (lane == 0) {
                D.lens_out[b] = new_len;
                D.qs_out[b] = q;
                D.status[b] = res;
            }
        }
        int cls = -1;
        if (new_len > 0 && new_len <= cap && q >= 0 && q < D.T.n_lex)
            cls = walk_class<true>(table, D.T.n_lex, D.T.n_lr, st, new_len, q, lane, s_ov, ptr);
        if (lane == 0) {
            s_cls = cls;
            if (cls < 0 && blockIdx.x == 0) atomicAdd(err, 1u);
        }
    }
    __syncthreads();
    return s_cls;
}

// psc_decode_step's first launch when its grid would not fit on the GPU at
// once: one wavefront per sequence advances it and writes the new state
// (the second launch is the fused step on the new states).
__global__ void __launch_bounds__(kWave)
advance_copy_kernel(DecodeArgs D) {
    __shared__ int32_t s_ov[kOverlay];
    const int b = blockIdx.x;
    const int lane = threadIdx.x;
    const int cap = D.cap;
    const int len = D.lens_in[b], q_in = D.qs_in[b];
    const int32_t *st = D.stacks_in + (int64_t)b * cap;
    int ptr, ov, q;
    const int res = advance_core(D.T, s_ov, st, len, q_in, D.tokens[b], cap, lane, ptr, ov, q);
    int32_t *dst = D.stacks_out + (int64_t)b * cap;
    const int keep = res == PSC_ADV_OK ? ptr : min(max(len, 0), cap);
    for (int k = lane; k < keep; k += kWave) dst[k] = st[k];
    for (int k = lane; k < ov; k += kWave) dst[ptr + k] = s_ov[k];
    if (lane == 0) {
        D.lens_out[b] = res == PSC_ADV_OK ? ptr + ov : len;
        D.qs_out[b] = q;
        D.status[b] = res;
    }
}

template <bool kBf16, bool kSliced>
__global__ void __launch_bounds__(kFusedBlock)
decode_fast_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                   const int32_t *__restrict__ ids, DecodeArgs D, int32_t W, uint32_t *__restrict__ out,
                   uint32_t *__restrict__ err, uint4 *__restrict__ logits) {
    const int b = blockIdx.y;
    const int cls = decode_block_class(table, D, b, err);
    fused_fast_apply<kBf16, kSliced>(cls, b, masks, mask_stride, ids, W, out, logits);
}

template <bool kBf16, bool kSliced>
__global__ void __launch_bounds__(kBlock)
decode_generic_kernel(const int32_t *__restrict__ table, const uint32_t *__restrict__ masks, int32_t mask_stride,
                      const int32_t *__restrict__ ids, DecodeArgs D, int32_t V, int32_t W,
                      uint32_t *__restrict__ out, uint32_t *__restrict__ err, void *__restrict__ logits) {
    const int b = blockIdx.y;
    const int cls = decode_block_class(table, D, b, err);
    fused_generic_apply<kBf16, kSliced>(cls, b, masks, mask_stride, ids, V, W, out, logits);
}

// Every predictor entry to the same value (psc_predictor_fill).
__global__ void __launch_bounds__(kBlock)
pred_fill_kernel(int32_t *__restrict__ pred, int64_t n, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) pred[i] = v;
}

psc_status device_fail(const char *what, hipError_t e) {
    set_error(std::string(what) + ": " + hipGetErrorString(e));
    return PSC_E_DEVICE;
}

psc_status check_bound(const psc_handle *h, const char *what) {
    if (!h) {
        set_error(std::string(what) + ": null handle");
        return PSC_E_INVALID_ARG;
    }
    if (!h->dev_base) {
        set_error(std::string(what) + ": device tables not bound");
        return PSC_E_NOT_BOUND;
    }
    return PSC_OK;
}

// The bound tables as the kernels read them; mstride is the mask row
// stride in words (flat) or the slices per row (sliced).
struct Bound {
    const int32_t *table;
    const uint32_t *masks;
    const int32_t *ids;
    int32_t mstride;
    uint32_t *err;
    int32_t *pred;
    bool sliced;
};

Bound bound(const psc_handle *h) {
    char *base = static_cast<char *>(h->dev_base);
    return Bound{reinterpret_cast<const int32_t *>(base + table_off(h->n_lex)),
                 reinterpret_cast<const uint32_t *>(base + h->mask_off),
                 reinterpret_cast<const int32_t *>(base + h->ids_off), h->sliced ? h->n_slices : h->mask_stride,
                 reinterpret_cast<uint32_t *>(base), reinterpret_cast<int32_t *>(base + h->pred_off), h->sliced};
}

psc_status check_states(const psc_handle *h, const int32_t *stacks, int32_t stride, int64_t n_stack,
                        const int32_t *stack_lens, const int32_t *lexer_states, int32_t B, const void *out,
                        const char *what) {
    if (psc_status st = check_bound(h, what)) return st;
    if (B < 0 || stride < 0 || n_stack < 0 || (B > 0 && (!stacks || !stack_lens || !lexer_states || !out))) {
        set_error(std::string(what) + ": null argument or negative size");
        return PSC_E_INVALID_ARG;
    }
    if (B > 65535) {
        set_error(std::string(what) + ": B > 65535");
        return PSC_E_INVALID_ARG;
    }
    return PSC_OK;
}

psc_status check_logits(const psc_handle *h, const void *logits, psc_dtype dtype, int32_t V, int32_t B,
                        const char *what) {
    if (dtype != PSC_F32 && dtype != PSC_BF16) {
        set_error(std::string(what) + ": bad dtype");
        return PSC_E_INVALID_ARG;
    }
    if (B > 0 && !logits) {
        set_error(std::string(what) + ": null logits");
        return PSC_E_INVALID_ARG;
    }
    if (V != h->V) {
        set_error(std::string(what) + ": V (" + std::to_string(V) + ") differs from the vocabulary size (" +
                  std::to_string(h->V) + ")");
        return PSC_E_INVALID_ARG;
    }
    return PSC_OK;
}

psc_status launched(const char *what) {
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail(what, e);
}

// The walk + gather for ragged (stride 0) or strided stacks.
psc_status launch_compute(const psc_handle *h, const int32_t *stacks, int32_t stride, int64_t n_stack,
                          const int32_t *stack_lens, const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                          void *stream, const char *what) {
    if (psc_status st = check_states(h, stacks, stride, n_stack, stack_lens, lexer_states, B, out_bitmask, what))
        return st;
    if (B == 0) return PSC_OK;
    const Bound T = bound(h);
    const int32_t W = h->W;
    const int vec4 = (W % 4 == 0) && ((reinterpret_cast<uintptr_t>(out_bitmask) & 15) == 0);
    dim3 grid((W + kCopyWordsPerBlock - 1) / kCopyWordsPerBlock, B);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (T.sliced)
        hipLaunchKernelGGL(walk_gather_kernel<true>, grid, dim3(kBlock), 0, s, T.table, T.masks, T.mstride, T.ids,
                           h->n_lex, h->n_lr, stacks, stride, n_stack, stack_lens, lexer_states, B, W, out_bitmask,
                           T.err, vec4);
    else
        hipLaunchKernelGGL(walk_gather_kernel<false>, grid, dim3(kBlock), 0, s, T.table, T.masks, T.mstride, T.ids,
                           h->n_lex, h->n_lr, stacks, stride, n_stack, stack_lens, lexer_states, B, W, out_bitmask,
                           T.err, vec4);
    return launched(what);
}

// The walk alone for ragged (stride 0) or strided stacks.
psc_status launch_classes(const psc_handle *h, const int32_t *stacks, int32_t stride, int64_t n_stack,
                          const int32_t *stack_lens, const int32_t *lexer_states, int32_t B, int32_t *out_classes,
                          void *stream, const char *what) {
    if (psc_status st = check_states(h, stacks, stride, n_stack, stack_lens, lexer_states, B, out_classes, what))
        return st;
    if (B == 0) return PSC_OK;
    const Bound T = bound(h);
    const int per_block = kBlock / kWave;
    hipLaunchKernelGGL(classes_kernel, dim3((B + per_block - 1) / per_block), dim3(kBlock), 0,
                       reinterpret_cast<hipStream_t>(stream), T.table, h->n_lex, h->n_lr, h->n_classes, stacks,
                       stride, n_stack, stack_lens, lexer_states, B, out_classes, T.err, T.pred);
    return launched(what);
}

// Words of the mask row per fused workgroup on the fast path.
int32_t fused_words_per_block(bool bf16) {
    return (kFusedBlock / kWave) * (bf16 ? ApplyGeom<true>::kWordsPerWave : ApplyGeom<false>::kWordsPerWave);
}

struct FastArgs {
    dim3 grid;
    hipStream_t s;
    Bound T;
    int32_t n_lex, n_lr, n_classes;
    const int32_t *stacks;
    int32_t stride;
    int64_t n_stack;
    const int32_t *lens, *qs;
    int32_t W;
    uint32_t *out;
    uint4 *logits;
    unsigned long long *tl;
};

template <bool kBf16, bool kSliced, bool kTl>
void launch_fast(bool spec, const FastArgs &F) {
    const Bound &T = F.T;
    if (spec)
        hipLaunchKernelGGL((fused_spec_kernel<kBf16, kSliced, kTl>), F.grid, dim3(kFusedBlock), 0, F.s, T.table,
                           T.masks, T.mstride, T.ids, F.n_lex, F.n_lr, F.n_classes, F.stacks, F.stride, F.n_stack,
                           F.lens, F.qs, F.W, F.out, T.err, T.pred, F.logits, F.tl);
    else
        hipLaunchKernelGGL((fused_fast_kernel<kBf16, kSliced, kTl>), F.grid, dim3(kFusedBlock), 0, F.s, T.table,
                           T.masks, T.mstride, T.ids, F.n_lex, F.n_lr, F.stacks, F.stride, F.n_stack, F.lens, F.qs,
                           F.W, F.out, T.err, F.logits, F.tl);
}

template <bool kBf16>
void launch_fast_dtype(bool spec, bool sliced, bool tl, const FastArgs &F) {
    if (sliced) {
        if (tl) launch_fast<kBf16, true, true>(spec, F);
        else launch_fast<kBf16, true, false>(spec, F);
    } else {
        if (tl) launch_fast<kBf16, false, true>(spec, F);
        else launch_fast<kBf16, false, false>(spec, F);
    }
}

// The single-launch step for ragged (stride 0) or strided stacks; with
// `tl` (fast path only) the timeline variant.
psc_status launch_fused(const psc_handle *h, const int32_t *stacks, int32_t stride, int64_t n_stack,
                        const int32_t *stack_lens, const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                        void *logits, psc_dtype dtype, int32_t V, void *stream, const char *what,
                        unsigned long long *tl = nullptr, int64_t n_tl = 0) {
    // out_bitmask may be null: the logits stand in for it in the null check
    if (psc_status st = check_states(h, stacks, stride, n_stack, stack_lens, lexer_states, B,
                                     out_bitmask ? static_cast<const void *>(out_bitmask) : logits, what))
        return st;
    if (psc_status st = check_logits(h, logits, dtype, V, B, what)) return st;
    const bool bf16 = dtype == PSC_BF16;
    const bool fast = (V % 32 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
    const int32_t W = h->W;
    if (tl) {
        const int64_t need = (int64_t)((W + fused_words_per_block(bf16) - 1) / fused_words_per_block(bf16)) * B *
                             (kFusedBlock / kWave);
        if (!fast || n_tl < need) {
            set_error(std::string(what) + ": the timeline needs the fast path (V % 32 == 0, 16-byte aligned "
                      "logits) and " + std::to_string(need) + " records");
            return PSC_E_INVALID_ARG;
        }
    }
    if (B == 0) return PSC_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const Bound T = bound(h);
    if (fast) {
        const FastArgs F{dim3((W + fused_words_per_block(bf16) - 1) / fused_words_per_block(bf16), B), s, T,
                         h->n_lex, h->n_lr, h->n_classes, stacks, stride, n_stack, stack_lens, lexer_states, W,
                         out_bitmask, reinterpret_cast<uint4 *>(logits), tl};
        const bool spec = (h->options & PSC_OPT_SPECULATE) != 0;
        if (bf16) launch_fast_dtype<true>(spec, T.sliced, tl != nullptr, F);
        else launch_fast_dtype<false>(spec, T.sliced, tl != nullptr, F);
    } else {
        dim3 grid((W + kGenWords - 1) / kGenWords, B);
#define PSC_GENERIC(BF, SL)                                                                                          \
    hipLaunchKernelGGL((fused_generic_kernel<BF, SL>), grid, dim3(kBlock), 0, s, T.table, T.masks, T.mstride, T.ids,  \
                       h->n_lex, h->n_lr, stacks, stride, n_stack, stack_lens, lexer_states, V, W, out_bitmask,     \
                       T.err, logits)
        if (bf16 && T.sliced) PSC_GENERIC(true, true);
        else if (bf16) PSC_GENERIC(true, false);
        else if (T.sliced) PSC_GENERIC(false, true);
        else PSC_GENERIC(false, false);
#undef PSC_GENERIC
    }
    return launched(what);
}

// The masked argmax for ragged (stride 0) or strided stacks.
// `records` is the per-sequence slot array (kArgmaxRecordWords uint64 per
// sequence, zero between calls); null selects the bound buffer's.
psc_status launch_argmax(const psc_handle *h, const int32_t *stacks, int32_t stride, int64_t n_stack,
                         const int32_t *stack_lens, const int32_t *lexer_states, int32_t B, const void *logits,
                         psc_dtype dtype, int32_t V, int32_t *out_tokens, void *stream, const char *what,
                         unsigned long long *records = nullptr) {
    if (psc_status st = check_states(h, stacks, stride, n_stack, stack_lens, lexer_states, B, out_tokens, what))
        return st;
    if (psc_status st = check_logits(h, logits, dtype, V, B, what)) return st;
    if (B == 0) return PSC_OK;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(h->dev_base);
    const Bound T = bound(h);
    const int fast = (V % 32 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
    const int32_t W = h->W;
    const int words_per_block = !fast ? kGenWords : fused_words_per_block(dtype == PSC_BF16);
    dim3 grid((W + words_per_block - 1) / words_per_block, B);
    if (!records) records = reinterpret_cast<unsigned long long *>(base + h->argmax_off);
#define PSC_ARGMAX(BF, SL)                                                                                           \
    hipLaunchKernelGGL((argmax_partial_kernel<BF, SL>), grid, dim3(kFusedBlock), 0, s, T.table, T.masks, T.mstride,   \
                       T.ids, h->n_lex, h->n_lr, stacks, stride, n_stack, stack_lens, lexer_states, V, W, T.err,    \
                       logits, fast, records, out_tokens)
    if (dtype == PSC_BF16 && T.sliced) PSC_ARGMAX(true, true);
    else if (dtype == PSC_BF16) PSC_ARGMAX(true, false);
    else if (T.sliced) PSC_ARGMAX(false, true);
    else PSC_ARGMAX(false, false);
#undef PSC_ARGMAX
    return launched(what);
}

// Per-device address of `scratch`, taken once per device (at the first
// bind on it, with that device current) and cleared there; null until then.
constexpr int kMaxDevices = 64;
std::atomic<unsigned long long *> g_scratch[kMaxDevices];
std::mutex g_scratch_mutex;

hipError_t scratch_setup(int device, hipStream_t s) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch[device].load(std::memory_order_acquire)) return hipSuccess;
    void *ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)kScratchSeqs * kArgmaxRecordWords;
    hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0, s,
                       static_cast<unsigned long long *>(ptr), n);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess) g_scratch[device].store(static_cast<unsigned long long *>(ptr), std::memory_order_release);
    return e;
}

constexpr int64_t kUnbounded = INT64_MAX;

psc_status check_dense(const int32_t *stacks, int32_t cap, const int32_t *lens, const int32_t *qs, int32_t B,
                       const char *what) {
    if (B < 0 || cap < 1 || (B > 0 && (!stacks || !lens || !qs))) {
        set_error(std::string(what) + ": null argument, B < 0 or cap < 1");
        return PSC_E_INVALID_ARG;
    }
    if ((int64_t)B * cap > ((int64_t)1 << 40)) {
        set_error(std::string(what) + ": B * cap too large");
        return PSC_E_INVALID_ARG;
    }
    return PSC_OK;
}

// The problem instance in the bound buffer, as the advance reads it.
AdvTables adv_tables(const psc_handle *h) {
    const char *base = static_cast<const char *>(h->dev_base);
    const int32_t *g = reinterpret_cast<const int32_t *>(base + h->gram_off);
    const psc::AdvanceLayout &L = h->adv;
    const int32_t *action = h->action_packed ? reinterpret_cast<const int32_t *>(base + h->packed_off) : g + L.action;
    return AdvTables{g + L.lex_next, g + L.lex_accept, g + L.ignored, action, g + L.go, g + L.prod_lhs,
                     g + L.prod_len, g + L.tok_off, reinterpret_cast<const uint8_t *>(base + h->vbytes_off),
                     h->n_lex, h->n_lr, L.n_term, L.n_nt, L.end_term, L.eos, h->V, h->action_packed ? 1 : 0,
                     h->has_closure ? reinterpret_cast<const int32_t *>(base + h->closure_off) : nullptr};
}

// Workgroups of 256 threads that fit on the current GPU at once: 8 per
// compute unit (4 SIMDs x 8 wavefronts; the fused kernels' registers allow
// it), from the device's compute-unit count.
int64_t resident_blocks() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    return (int64_t)cus * 8;
}

bool ranges_overlap(const void *a, const void *b, size_t n) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + n && y < x + n;
}

}  // namespace

extern "C" psc_status psc_bind_device_ex(psc_handle *h, void *dev_buf, size_t nbytes, uint32_t flags,
                                         void *stream) {
    if (!h || !dev_buf || (reinterpret_cast<uintptr_t>(dev_buf) & 255) != 0) {
        set_error("psc_bind_device: null handle/buffer or buffer not 256-byte aligned");
        return PSC_E_INVALID_ARG;
    }
    if (flags & ~(uint32_t)(PSC_BIND_FLAT | PSC_BIND_SLICED) || flags == (PSC_BIND_FLAT | PSC_BIND_SLICED)) {
        set_error("psc_bind_device: unknown flags");
        return PSC_E_INVALID_ARG;
    }
    const DeviceLayout L = device_layout(*h, flags);
    if (nbytes < L.total) {
        set_error("psc_bind_device: buffer too small (" + std::to_string(nbytes) + " < " + std::to_string(L.total) +
                  ")");
        return PSC_E_INVALID_ARG;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(dev_buf);
    // the tables derived at bind time, on the host first
    std::vector<int32_t> packed, closure, blocks;
    bool is_packed = false;
    try {
        is_packed = packed_action(*h, packed);
        goto_closure(*h, closure);
        start_blocks(*h, blocks);
    } catch (const std::bad_alloc &) {
        set_error("psc_bind_device: out of host memory");
        return PSC_E_OOM;
    }
    hipError_t e = hipMemsetAsync(base, 0, kStartBlockOff, s);
    auto put = [&](size_t off, const void *src, size_t n) {
        if (e == hipSuccess && n) e = hipMemcpyAsync(base + off, src, n, hipMemcpyHostToDevice, s);
    };
    put(kStartBlockOff, blocks.data(), blocks.size() * sizeof(int32_t));
    if (e == hipSuccess) e = hipMemsetAsync(base + L.argmax, 0, kArgmaxBytes, s);
    put(L.table, h->table.data(), h->table.size() * sizeof(int32_t));
    if (L.sliced) {
        put(L.masks, h->slices.data(), h->slices.size() * sizeof(uint32_t));
        put(L.ids, h->slice_ids.data(), h->slice_ids.size() * sizeof(int32_t));
    } else {
        put(L.masks, h->masks.data(), h->masks.size() * sizeof(uint32_t));
    }
    put(L.gram, h->gram.data(), h->gram.size() * sizeof(int32_t));
    put(L.vbytes, h->vbytes.data(), h->vbytes.size());
    if (is_packed) put(L.packed, packed.data(), packed.size() * sizeof(int32_t));
    if (!closure.empty()) put(L.closure, closure.data(), closure.size() * sizeof(int32_t));
    // the predictor starts empty (-1 in every entry)
    if (e == hipSuccess)
        e = hipMemsetAsync(base + L.pred, 0xFF, (size_t)start_block_count(h->n_lex) * kPredInts * sizeof(int32_t), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    int device = -1;
    if (e == hipSuccess) e = hipGetDevice(&device);
    if (e == hipSuccess) e = scratch_setup(device, s);
    if (e != hipSuccess) return device_fail("psc_bind_device", e);
    h->device = device;
    h->dev_base = dev_buf;
    h->dev_bytes = nbytes;
    h->sliced = L.sliced;
    h->mask_off = L.masks;
    h->ids_off = L.ids;
    h->gram_off = L.gram;
    h->vbytes_off = L.vbytes;
    h->argmax_off = L.argmax;
    h->packed_off = L.packed;
    h->action_packed = is_packed;
    h->closure_off = L.closure;
    h->has_closure = !closure.empty();
    h->pred_off = L.pred;
    h->info.bound_mask_layout = L.sliced ? PSC_BIND_SLICED : PSC_BIND_FLAT;
    return PSC_OK;
}

extern "C" psc_status psc_bind_device(psc_handle *h, void *dev_buf, size_t nbytes, void *stream) {
    return psc_bind_device_ex(h, dev_buf, nbytes, 0, stream);
}

extern "C" psc_status psc_compute_masks(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                        const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                                        void *stream) {
    return launch_compute(h, stacks, 0, kUnbounded, stack_lens, lexer_states, B, out_bitmask, stream,
                          "psc_compute_masks");
}

extern "C" psc_status psc_compute_masks_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                          const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                          uint32_t *out_bitmask, void *stream) {
    return launch_compute(h, stacks, 0, n_stack, stack_lens, lexer_states, B, out_bitmask, stream,
                          "psc_compute_masks_n");
}

extern "C" psc_status psc_compute_classes(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                          const int32_t *lexer_states, int32_t B, int32_t *out_classes,
                                          void *stream) {
    return launch_classes(h, stacks, 0, kUnbounded, stack_lens, lexer_states, B, out_classes, stream,
                          "psc_compute_classes");
}

extern "C" psc_status psc_compute_classes_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                            const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                            int32_t *out_classes, void *stream) {
    return launch_classes(h, stacks, 0, n_stack, stack_lens, lexer_states, B, out_classes, stream,
                          "psc_compute_classes_n");
}

extern "C" psc_status psc_compute_classes_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                                const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                                int32_t *out_classes, void *stream) {
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_compute_classes_dense"))
        return st;
    return launch_classes(h, stacks, cap, kUnbounded, stack_lens, lexer_states, B, out_classes, stream,
                          "psc_compute_classes_dense");
}

extern "C" psc_status psc_compute_and_apply(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                            const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                                            void *logits, psc_dtype dtype, int32_t V, void *stream) {
    return launch_fused(h, stacks, 0, kUnbounded, stack_lens, lexer_states, B, out_bitmask, logits, dtype, V, stream,
                        "psc_compute_and_apply");
}

extern "C" psc_status psc_compute_and_apply_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                              const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                              uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                              void *stream) {
    return launch_fused(h, stacks, 0, n_stack, stack_lens, lexer_states, B, out_bitmask, logits, dtype, V, stream,
                        "psc_compute_and_apply_n");
}

extern "C" int64_t psc_timeline_records(const psc_handle *h, int32_t B, psc_dtype dtype) {
    if (!h || B < 0) return 0;
    const int32_t per = fused_words_per_block(dtype == PSC_BF16);
    return (int64_t)((h->W + per - 1) / per) * B * (kFusedBlock / kWave);
}

extern "C" psc_status psc_compute_and_apply_timeline(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                                     const int32_t *stack_lens, const int32_t *lexer_states,
                                                     int32_t B, uint32_t *out_bitmask, void *logits,
                                                     psc_dtype dtype, int32_t V, uint64_t *records,
                                                     int64_t n_records, void *stream) {
    if (!records) {
        set_error("psc_compute_and_apply_timeline: null records");
        return PSC_E_INVALID_ARG;
    }
    return launch_fused(h, stacks, 0, n_stack, stack_lens, lexer_states, B, out_bitmask, logits, dtype, V, stream,
                        "psc_compute_and_apply_timeline", reinterpret_cast<unsigned long long *>(records), n_records);
}

extern "C" psc_status psc_compute_masks_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                              const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                              uint32_t *out_bitmask, void *stream) {
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_compute_masks_dense")) return st;
    return launch_compute(h, stacks, cap, kUnbounded, stack_lens, lexer_states, B, out_bitmask, stream,
                          "psc_compute_masks_dense");
}

extern "C" psc_status psc_compute_and_apply_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                                  const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                                  uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                                  void *stream) {
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_compute_and_apply_dense"))
        return st;
    return launch_fused(h, stacks, cap, kUnbounded, stack_lens, lexer_states, B, out_bitmask, logits, dtype, V,
                        stream, "psc_compute_and_apply_dense");
}

extern "C" psc_status psc_compute_and_argmax(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                             const int32_t *lexer_states, int32_t B, const void *logits,
                                             psc_dtype dtype, int32_t V, int32_t *out_tokens, void *stream) {
    return launch_argmax(h, stacks, 0, kUnbounded, stack_lens, lexer_states, B, logits, dtype, V, out_tokens, stream,
                         "psc_compute_and_argmax");
}

extern "C" psc_status psc_compute_and_argmax_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                               const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                               const void *logits, psc_dtype dtype, int32_t V, int32_t *out_tokens,
                                               void *stream) {
    return launch_argmax(h, stacks, 0, n_stack, stack_lens, lexer_states, B, logits, dtype, V, out_tokens, stream,
                         "psc_compute_and_argmax_n");
}

extern "C" psc_status psc_compute_and_argmax_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                                   const int32_t *stack_lens, const int32_t *lexer_states,
                                                   int32_t B, const void *logits, psc_dtype dtype, int32_t V,
                                                   int32_t *out_tokens, void *stream) {
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_compute_and_argmax_dense"))
        return st;
    return launch_argmax(h, stacks, cap, kUnbounded, stack_lens, lexer_states, B, logits, dtype, V, out_tokens,
                         stream, "psc_compute_and_argmax_dense");
}

extern "C" psc_status psc_compute_and_argmax_noalloc(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                                    const int32_t *stack_lens, const int32_t *lexer_states,
                                                    int32_t B, const void *logits, psc_dtype dtype, int32_t V,
                                                    int32_t *out_tokens, void *stream) {
    const char *what = "psc_compute_and_argmax_noalloc";
    if (psc_status st = check_bound(h, what)) return st;
    if (B > kScratchSeqs) {
        set_error(std::string(what) + ": B > " + std::to_string(kScratchSeqs) +
                  " (the fixed record array holds that many sequences)");
        return PSC_E_INVALID_ARG;
    }
    unsigned long long *records =
        h->device >= 0 && h->device < kMaxDevices ? g_scratch[h->device].load(std::memory_order_acquire) : nullptr;
    if (!records) {
        set_error(std::string(what) + ": no record array on the bound device");
        return PSC_E_NOT_BOUND;
    }
    return launch_argmax(h, stacks, 0, n_stack, stack_lens, lexer_states, B, logits, dtype, V, out_tokens, stream,
                         what, records);
}

extern "C" psc_status psc_set_options(psc_handle *h, uint32_t options) {
    if (!h || (options & ~(uint32_t)PSC_OPT_SPECULATE)) {
        set_error("psc_set_options: null handle or unknown option");
        return PSC_E_INVALID_ARG;
    }
    h->options = options;
    return PSC_OK;
}

extern "C" psc_status psc_predictor_fill(const psc_handle *h, int32_t cls, void *stream) {
    if (psc_status st = check_bound(h, "psc_predictor_fill")) return st;
    if (cls < -1 || cls >= h->n_classes) {
        set_error("psc_predictor_fill: class out of range");
        return PSC_E_INVALID_ARG;
    }
    const int64_t n = (int64_t)start_block_count(h->n_lex) * kPredInts;
    hipLaunchKernelGGL(pred_fill_kernel, dim3((unsigned)std::min<int64_t>((n + kBlock - 1) / kBlock, 4096)),
                       dim3(kBlock), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<int32_t *>(static_cast<char *>(h->dev_base) + h->pred_off), n, cls);
    return launched("psc_predictor_fill");
}

extern "C" psc_status psc_predictor_updates(const psc_handle *h, uint32_t *out, int32_t reset, void *stream) {
    if (!out) {
        set_error("psc_predictor_updates: null argument");
        return PSC_E_INVALID_ARG;
    }
    if (psc_status st = check_bound(h, "psc_predictor_updates")) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    uint32_t *ctr = static_cast<uint32_t *>(h->dev_base) + kCounterPredUpdates;
    hipError_t e = hipMemcpyAsync(out, ctr, sizeof(uint32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess && reset) e = hipMemsetAsync(ctr, 0, sizeof(uint32_t), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    return e == hipSuccess ? PSC_OK : device_fail("psc_predictor_updates", e);
}

extern "C" psc_status psc_state_reset(const psc_handle *h, int32_t *stacks, int32_t cap, int32_t *stack_lens,
                                      int32_t *lexer_states, int32_t B, void *stream) {
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_state_reset")) return st;
    if (!h) {
        set_error("psc_state_reset: null handle");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0) return PSC_OK;
    hipLaunchKernelGGL(reset_kernel, dim3((B + kBlock - 1) / kBlock), dim3(kBlock), 0,
                       reinterpret_cast<hipStream_t>(stream), stacks, cap, stack_lens, lexer_states, B);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail("psc_state_reset", e);
}

extern "C" psc_status psc_advance(const psc_handle *h, int32_t *stacks, int32_t cap, int32_t *stack_lens,
                                  int32_t *lexer_states, int32_t B, const int32_t *tokens, int32_t *status,
                                  void *stream) {
    if (psc_status st = check_bound(h, "psc_advance")) return st;
    if (psc_status st = check_dense(stacks, cap, stack_lens, lexer_states, B, "psc_advance")) return st;
    if (B > 0 && (!tokens || !status)) {
        set_error("psc_advance: null tokens or status");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0) return PSC_OK;
    const AdvTables T = adv_tables(h);
    hipLaunchKernelGGL(advance_kernel, dim3(B), dim3(kWave), 0,
                       reinterpret_cast<hipStream_t>(stream), T, stacks, cap, stack_lens, lexer_states, B, tokens,
                       status);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail("psc_advance", e);
}

extern "C" psc_status psc_decode_step(const psc_handle *h, const int32_t *stacks_in, const int32_t *lens_in,
                                      const int32_t *qs_in, int32_t *stacks_out, int32_t *lens_out, int32_t *qs_out,
                                      int32_t cap, int32_t B, const int32_t *tokens, int32_t *status,
                                      uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                      void *stream) {
    const char *what = "psc_decode_step";
    if (psc_status st = check_bound(h, what)) return st;
    if (psc_status st = check_dense(stacks_in, cap, lens_in, qs_in, B, what)) return st;
    if (psc_status st = check_dense(stacks_out, cap, lens_out, qs_out, B, what)) return st;
    if (B > 0 && (!tokens || !status || !logits || (dtype != PSC_F32 && dtype != PSC_BF16))) {
        set_error("psc_decode_step: null tokens, status or logits, or bad dtype");
        return PSC_E_INVALID_ARG;
    }
    if (V != h->V) {
        set_error("psc_decode_step: V differs from the vocabulary size");
        return PSC_E_INVALID_ARG;
    }
    if (B > 65535) {
        set_error("psc_decode_step: B > 65535");
        return PSC_E_INVALID_ARG;
    }
    if (B == 0) return PSC_OK;
    const size_t n_st = (size_t)B * cap * sizeof(int32_t), n_b = (size_t)B * sizeof(int32_t);
    if (ranges_overlap(stacks_in, stacks_out, n_st) || ranges_overlap(lens_in, lens_out, n_b) ||
        ranges_overlap(qs_in, qs_out, n_b)) {
        set_error("psc_decode_step: the input and output states overlap");
        return PSC_E_INVALID_ARG;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char *base = static_cast<char *>(h->dev_base);
    const Bound T = bound(h);
    const DecodeArgs D{adv_tables(h), stacks_in, lens_in, qs_in, stacks_out, lens_out, qs_out, tokens, status, cap};
    const int32_t W = h->W;
    const bool bf16 = dtype == PSC_BF16;
    const bool fast = (V % 32 == 0) && ((reinterpret_cast<uintptr_t>(logits) & 15) == 0);
    // When the fused grid does not fit on the GPU at once, workgroups that
    // start late would repeat the advance after the early ones finished:
    // then the advance runs once per sequence in a launch of its own and the
    // fused step follows on the new states (same results).
    const int words_per_block = !fast ? kGenWords
                                      : (kFusedBlock / kWave) * (bf16 ? ApplyGeom<true>::kWordsPerWave
                                                                      : ApplyGeom<false>::kWordsPerWave);
    const int64_t n_blocks = (int64_t)((W + words_per_block - 1) / words_per_block) * B;
    if (n_blocks > resident_blocks()) {
        hipLaunchKernelGGL(advance_copy_kernel, dim3(B), dim3(kWave), 0, s, D);
        hipError_t e0 = hipGetLastError();
        if (e0 != hipSuccess) return device_fail(what, e0);
        return launch_fused(h, stacks_out, cap, kUnbounded, lens_out, qs_out, B, out_bitmask, logits, dtype, V, stream,
                            what);
    }
    if (fast) {
        const int words_per_block = (kFusedBlock / kWave) * (bf16 ? ApplyGeom<true>::kWordsPerWave
                                                                  : ApplyGeom<false>::kWordsPerWave);
        dim3 grid((W + words_per_block - 1) / words_per_block, B);
#define PSC_DECODE_FAST(BF, SL)                                                                                      \
    hipLaunchKernelGGL((decode_fast_kernel<BF, SL>), grid, dim3(kFusedBlock), 0, s, T.table, T.masks, T.mstride, T.ids, \
                       D, W, out_bitmask, T.err, reinterpret_cast<uint4 *>(logits))
        if (bf16 && T.sliced) PSC_DECODE_FAST(true, true);
        else if (bf16) PSC_DECODE_FAST(true, false);
        else if (T.sliced) PSC_DECODE_FAST(false, true);
        else PSC_DECODE_FAST(false, false);
#undef PSC_DECODE_FAST
    } else {
        dim3 grid((W + kGenWords - 1) / kGenWords, B);
#define PSC_DECODE_GEN(BF, SL)                                                                                       \
    hipLaunchKernelGGL((decode_generic_kernel<BF, SL>), grid, dim3(kBlock), 0, s, T.table, T.masks, T.mstride, T.ids,   \
                       D, V, W, out_bitmask, T.err, logits)
        if (bf16 && T.sliced) PSC_DECODE_GEN(true, true);
        else if (bf16) PSC_DECODE_GEN(true, false);
        else if (T.sliced) PSC_DECODE_GEN(false, true);
        else PSC_DECODE_GEN(false, false);
#undef PSC_DECODE_GEN
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? PSC_OK : device_fail(what, e);
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
        const int64_t words_per_wave = bf16 ? ApplyGeom<true>::kWordsPerWave : ApplyGeom<false>::kWordsPerWave;
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
