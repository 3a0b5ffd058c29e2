// Internal layout shared by the host construction (psc_build.cpp) and the
// device entry points (psc_device.hip).  Not part of the public ABI.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/psc.h"

namespace psc {

// A reference to an automaton state as stored in the flat table:
//   ref >= 0 : the state's row starts at int32 offset (ref & ~1) of the
//              table; bit 0 set means the row is dense over the stack
//              alphabet, clear means sparse (sorted (symbol, ref) pairs).
//   ref <  0 : the state is determined -- every stack continuation ends in
//              the same class -- and that class is (-ref - 1).
// Row header (4 int32): end_class, n_edges (sparse) or -1 (dense),
// default_ref (sparse), skip.  Sparse rows follow with n_edges pairs
// (symbol, ref); dense rows with n_lr_states refs indexed by symbol.
// A sparse row with n_edges == 0 heads a skip chain: every symbol leads to
// the default and the class cannot change, so skip = L >= 1 symbols are
// consumed at once and default_ref is the state reached after them (if the
// stack ends inside the chain, the class is this row's end_class).
// Rows start at even offsets so a pair is one aligned 8-byte load.
constexpr int kRowHeader = 4;
constexpr int kSparseMax = 62;      // header + edges in one wavefront-wide load
constexpr int kTablePad = 2 * 64 + kRowHeader;  // a row load reads 128 int32 speculatively

inline bool ref_is_class(int32_t ref) { return ref < 0; }
inline int32_t ref_class(int32_t ref) { return -ref - 1; }
inline int32_t class_ref(int32_t cls) { return -cls - 1; }
inline bool ref_is_dense(int32_t ref) { return (ref & 1) != 0; }
inline int32_t ref_offset(int32_t ref) { return ref & ~1; }

// Device buffer layout (offsets in bytes from the bound base):
//   [0, 256)                   uint32 error counter (+ padding)
//   [kTableOff, ...)           int32 table: start refs [n_lex], rows, pad
//   [mask_off, ...)            uint32 masks [n_classes][mask_stride] (256-B aligned)
constexpr size_t kTableOff = 256;

}  // namespace psc

struct psc_handle {
    int32_t V = 0, W = 0, mask_stride = 0, n_lex = 0, n_lr = 0, n_classes = 0;
    std::vector<int32_t> table;    // start refs then rows then padding
    std::vector<uint32_t> masks;   // [n_classes][mask_stride]
    psc_info_t info{};
    // device binding (caller-owned memory)
    void *dev_base = nullptr;
    size_t dev_bytes = 0;
    size_t mask_off = 0;
    size_t device_bytes_needed() const;
};

namespace psc {
void set_error(const std::string &msg);
}
