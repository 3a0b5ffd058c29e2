// Internal layout shared by the host construction (psc_build.cpp) and the
// device entry points (psc_device.hip).  Not part of the public ABI.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/psc.h"

namespace psc {

// A reference to an automaton state as stored in the flat table:
//   ref >= 0 : the state's row or chain entry starts at int32 offset
//              (ref & ~3) of the table; the low two bits give its kind:
//              0 sparse row, 1 dense row, 2 chain entry.
//   ref <  0 : the state is determined -- every stack continuation ends in
//              the same class -- and that class is (-ref - 1).
// Dense rows have a 4-int32 header (end_class, -1, default_ref, 0) and then
// n_lr_states entries (ref, skip) indexed by symbol.  Sparse rows are 16 bytes per lane of
// one wavefront-wide load: (end_class, n_edges, 0, 0), (kSymNone,
// default_ref, default_skip, 0), then n_edges entries (symbol, ref, skip, 0)
// sorted by symbol.  A skip (chain_skip) is set when the ref is a chain entry
// from which k >= 1 wildcard entries lead to the chain's jump: the walk may
// then read those k symbols without a load (checking only that they are in
// range) and go on at the jump's target, as the chain would.
//
// Chains: a state with at most two explicit edges (an edge-free state
// included) is one 16-byte entry of a chain, so that a walk through a run
// of such "thin" states costs one load per up to kChainMax symbols instead
// of one per symbol:
//   x = a | (b << 16)  a: the symbol that moves on to the next entry of the
//                      chain (kSymWild: any symbol), or kSymJump;
//                      b: the other explicit edge's symbol, or kSymNone;
//   y = ref on b;  z = ref on any other symbol (for kSymJump: the state the
//   chain continues with, reached without reading a symbol);  w = the
//   state's end_class (the class when the stack ends before it reads).
// A chain holds at most kChainMax states and ends with a kSymJump entry, so
// 64 consecutive entries read from any state of it include that entry.  A
// chain of fewer than kChainReach states is followed, before its jump, by
// copies of the thin states its last state continues into (their entries,
// never pointed at by a ref), up to kChainReach entries in all.
// Rows and entries start at multiples of 4 int32 (16-byte aligned).
constexpr int kRowHeader = 4;       // dense rows
constexpr int kSparseHeader = 8;    // sparse rows: two 16-byte header entries
constexpr int kSparseEdge = 4;      // int32 per sparse entry
constexpr int kSparseMax = 62;      // header + edges in one wavefront-wide load
constexpr int kChainMax = 63;
constexpr int kChainReach = 16;     // entries a chain is extended to with copies of its continuation
constexpr int kChainEntry = 4;      // int32 per entry
constexpr int32_t kSymNone = 0xFFFF, kSymWild = 0xFFFE, kSymJump = 0xFFFD;
constexpr int kMaxChainAlphabet = 0xFFFD;   // chains need every symbol < kSymJump
constexpr int kRefDense = 1, kRefChain = 2;
// a walk step reads 64 lanes x 16 bytes from a chain entry speculatively
constexpr int kTablePad = 64 * kChainEntry + kRowHeader;

// A skip: k (1..kSkipMax) wildcard entries, then the jump's target ref R,
// packed as k << 27 | (R + 2^26); kNoSkip when there is none or R does not fit.
constexpr int32_t kNoSkip = -1;
constexpr int kSkipMax = 15;
inline int32_t skip_encode(int k, int32_t target) {
    if (k < 1 || k > kSkipMax || target < -(1 << 26) || target >= (1 << 26)) return kNoSkip;
    return (int32_t)(((uint32_t)k << 27) | (uint32_t)(target + (1 << 26)));
}

inline bool ref_is_class(int32_t ref) { return ref < 0; }
inline int32_t ref_class(int32_t ref) { return -ref - 1; }
inline int32_t class_ref(int32_t cls) { return -cls - 1; }
inline bool ref_is_dense(int32_t ref) { return (ref & 3) == kRefDense; }
inline bool ref_is_chain(int32_t ref) { return (ref & 3) == kRefChain; }
inline int32_t ref_offset(int32_t ref) { return ref & ~3; }

// The skip of `ref` in a table of n int32 (kNoSkip unless ref is a chain
// entry followed, from itself, by 1..kSkipMax wildcard entries and the jump).
inline int32_t chain_skip(const int32_t *t, int64_t n, int32_t ref) {
    if (ref < 0 || !ref_is_chain(ref)) return kNoSkip;
    const int64_t p = ref_offset(ref);
    int k = 0;
    while (k <= kSkipMax && p + kChainEntry * k < n && (t[p + kChainEntry * k] & 0xFFFF) == kSymWild) k++;
    const int64_t j = p + kChainEntry * k;
    if (k < 1 || k > kSkipMax || j + 2 >= n || (t[j] & 0xFFFF) != kSymJump) return kNoSkip;
    return skip_encode(k, t[j + 2]);
}

// The problem instance as the device advance of prefix states reads it: one
// int32 blob, sections at these int32 offsets, plus the vocabulary bytes.
struct AdvanceLayout {
    int64_t lex_next = 0;   // [n_lex][256]
    int64_t lex_accept = 0; // [n_lex]
    int64_t ignored = 0;    // [n_term] 0/1
    int64_t action = 0;     // [n_lr][n_term]
    int64_t go = 0;         // [n_lr][n_nt]
    int64_t prod_lhs = 0;   // [n_prod]
    int64_t prod_len = 0;   // [n_prod]
    int64_t tok_off = 0;    // [V + 1] byte offsets of the spellings
    int32_t n_term = 0, n_nt = 0, end_term = 0, eos = -1;
};

// Device buffer layout (offsets in bytes from the bound base; device_layout
// computes them):
//   [0, 256)                   uint32 counters: [0] inputs rejected by a walk (range
//                              faults), [1] updates of the class predictor (+ padding)
//   [256, table_off(n_lex))    start blocks [min(n_lex, kMaxStartBlocks)][64 lanes][4] int32: block q holds the
//                              first walk step's wavefront load from start[q] (the 64
//                              chain entries, or the sparse row's header and entries), so
//                              that it is fetched together with the stack instead of after it
//   [table_off(n_lex), ...)    int32 table: start refs [n_lex], rows, pad
//   [mask_off, ...)            flat layout: uint32 masks [n_classes][mask_stride] (256-B aligned);
//                              sliced layout: uint32 slices [n_unique_slices][64], then
//                              int32 slice ids [n_classes][n_slices] at ids_off (row c of
//                              the flat table is slices[ids[c][0]], slices[ids[c][1]], ...)
//   [gram_off, ...)            int32 advance blob (AdvanceLayout)
//   [vbytes_off, ...)          uint8 vocabulary bytes
//   [argmax_off, ...)          masked argmax: [65536] records of 128 bytes, each a uint64
//                              slot then a uint32 arrival counter (zero between calls)
//   [packed_off, ...)          int32 ACTION with packed reductions (packed_action)
//   [closure_off, ...)         int32 unit-reduction closure of GOTO (goto_closure), when it fits
//   [pred_off, ...)            int32 class predictor [start_block_count(n_lex)][64][2]: for
//                              lexer state q and the way a walk's first step from start[q]
//                              left the start block (lane, kind), the class such a walk last
//                              reached; -1 = none
constexpr size_t kStartBlockOff = 256;
constexpr int kCounterFaults = 0, kCounterPredUpdates = 1;
constexpr int kSliceWords = 64;           // words per slice of a mask row (the sliced layout)
constexpr int kPredInts = 64 * 2;         // predictor slots per lexer state
constexpr int kStartBlockInts = 64 * 4;   // one 16-byte vector per lane
// Lexer states q < kMaxStartBlocks have a start block (at most 4 MB); a walk
// from a higher one reads start[q]'s row after start[q], as any other row.
constexpr int32_t kMaxStartBlocks = 4096;
constexpr int32_t start_block_count(int32_t n_lex) { return n_lex < kMaxStartBlocks ? n_lex : kMaxStartBlocks; }
constexpr size_t table_off(int32_t n_lex) {
    return kStartBlockOff + (size_t)start_block_count(n_lex) * kStartBlockInts * sizeof(int32_t);
}
constexpr size_t kArgmaxSlots = 65536;
constexpr size_t kArgmaxRecordWords = 16;   // uint64 words per record: one 128-byte cache line
constexpr size_t kArgmaxBytes = kArgmaxSlots * kArgmaxRecordWords * sizeof(unsigned long long);

}  // namespace psc

struct psc_handle {
    int32_t V = 0, W = 0, mask_stride = 0, n_lex = 0, n_lr = 0, n_classes = 0;
    std::vector<int32_t> table;    // start refs, rows, chains, padding
    int64_t rows_off = 0, chains_off = 0, table_end = 0;   // regions of the table (int32 offsets)
    std::vector<uint32_t> masks;   // [n_classes][mask_stride]
    std::vector<int32_t> gram;     // advance blob
    std::vector<uint8_t> vbytes;   // vocabulary bytes (at least 1)
    psc::AdvanceLayout adv;
    psc_info_t info{};
    // the mask table cut into kSliceWords-word slices, each distinct slice
    // stored once (slice_masks): n_slices = mask_stride / kSliceWords per row
    std::vector<uint32_t> slices;  // [n_unique_slices][kSliceWords]
    std::vector<int32_t> slice_ids;   // [n_classes][n_slices]
    int32_t n_slices = 0, n_unique_slices = 0;
    // device binding (caller-owned memory)
    void *dev_base = nullptr;
    size_t dev_bytes = 0;
    int device = -1;               // the HIP device current at bind time
    size_t mask_off = 0, ids_off = 0, gram_off = 0, vbytes_off = 0, argmax_off = 0, packed_off = 0,
           closure_off = 0, pred_off = 0;
    bool sliced = false;           // the bound mask table is the sliced layout
    uint32_t options = 0;          // PSC_OPT_* (psc_set_options)
    bool action_packed = false;    // the device ACTION copy carries each reduction's length and lhs
    bool has_closure = false;      // the device holds the unit-reduction closure of GOTO
    size_t device_bytes_needed(uint32_t flags = 0) const;
};

namespace psc {
void set_error(const std::string &msg);
// ACTION as the device advance reads it: a reduction's entry carries the
// production's length and left-hand side, kind | len << 2 | lhs << 10, so a
// reduction needs no second table read.  Returns false (and leaves `out`
// empty) when some production does not fit (length > 255 or lhs >= 2^21).
bool packed_action(const psc_handle &h, std::vector<int32_t> &out);
// GOTO followed by the unit reductions the lookahead then selects:
// closure[(s * n_nt + A) * n_term + t] is the state on top after a reduction
// to A returns to state s with lookahead t, GOTO[s][A] pushed and every
// following reduction by a one-symbol production done (each pops the state
// just pushed and pushes GOTO[s][B], so s stays below); -1 where a GOTO in
// that run is missing.  A run longer than n_nt (a cycle of unit
// productions) is left undone: the entry is GOTO[s][A].  Only built when it
// takes at most kClosureMaxBytes.
constexpr size_t kClosureMaxBytes = 64u << 20;
size_t goto_closure_bytes(const psc_handle &h);
void goto_closure(const psc_handle &h, std::vector<int32_t> &out);
// The start blocks, [start_block_count(n_lex)][kStartBlockInts]: block q is what a walk's
// first step from start[q] loads, one 16-byte vector per lane (a chain
// entry's 64 entries, or a sparse row's header and entries, as they are);
// zeros for a determined start or a dense row, which the walk does not read.
void start_blocks(const psc_handle &h, std::vector<int32_t> &out);
// The input checks of psc_build (ids in range, spellings), for loaded tables.
psc_status check_instance(const psc_grammar *g, const psc_vocab *v, std::string *msg);
// Cut the mask table into kSliceWords-word slices and keep each distinct
// slice once (h.slices, h.slice_ids); fills the sliced-layout fields of h.info.
void slice_masks(psc_handle &h);
// Byte offsets of every region of the bound buffer for the mask layout that
// `flags` selects (PSC_BIND_FLAT or PSC_BIND_SLICED; 0 = the default).
struct DeviceLayout {
    bool sliced;
    size_t table, masks, ids, gram, vbytes, argmax, packed, closure, pred, total;
};
DeviceLayout device_layout(const psc_handle &h, uint32_t flags);
}
