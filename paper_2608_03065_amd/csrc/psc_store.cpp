// Persistence of a built classifier: psc_save / psc_load.
//
// The construction (Algorithm 1) runs once per (grammar, vocabulary) pair and
// can take minutes for programming-language grammars (Tab. preprocess), so
// its result is stored and reloaded.  The file holds everything a handle
// needs -- the classifier table, the mask table and the problem instance the
// device advance reads -- in four checksummed sections; the larger ones are
// deflate-compressed.
//
// Format (little-endian, this library's struct layouts, version-checked):
//   FileHeader
//   4 x { SectionHeader, stored bytes }   tags TABL, MASK, GRAM, VBYT
// A loaded handle is untrusted input to the GPU kernels: before it is
// accepted, every ref of the classifier table is checked to name a row or a
// chain entry of the right kind or a class, chains must end within one
// wavefront load, and the problem instance passes psc_build's input checks.
#include <zlib.h>

#include <cstdio>
#include <cstring>
#include <exception>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "psc_internal.hpp"

using namespace psc;

namespace {

constexpr char kMagic[4] = {'P', 'S', 'C', 'B'};
constexpr uint32_t kVersion = 3;   // 3: row entries carry skips
constexpr uint32_t kCodecRaw = 0, kCodecZlib = 1;
constexpr uint64_t kMaxSection = 1ull << 40;      // sanity bound on a section's size
constexpr size_t kCompressAbove = 1 << 16;        // smaller sections are stored raw

constexpr uint32_t tag(const char (&t)[5]) {
    return (uint32_t)t[0] | (uint32_t)t[1] << 8 | (uint32_t)t[2] << 16 | (uint32_t)t[3] << 24;
}

struct FileHeader {
    char magic[4];
    uint32_t version;
    uint32_t header_bytes;
    uint32_t n_sections;
    int32_t V, W, mask_stride, n_lex, n_lr, n_classes;
    int64_t rows_off, chains_off, table_end;
    psc_info_t info;
    AdvanceLayout adv;
};

struct SectionHeader {
    uint32_t tag;
    uint32_t codec;
    uint64_t raw_bytes;
    uint64_t stored_bytes;
    uint64_t checksum;   // FNV-1a 64 of the raw bytes
};

uint64_t fnv1a(const void *p, size_t n) {
    const uint8_t *b = static_cast<const uint8_t *>(p);
    uint64_t h = 0xcbf29ce484222325ull;
    for (size_t i = 0; i < n; i++) h = (h ^ b[i]) * 0x100000001b3ull;
    return h;
}

struct StoreError {
    psc_status code;
    std::string msg;
};

[[noreturn]] void fail(psc_status c, const std::string &m) { throw StoreError{c, m}; }

struct File {
    FILE *f = nullptr;
    ~File() {
        if (f) fclose(f);
    }
};

void write_all(FILE *f, const void *p, size_t n) {
    if (n && fwrite(p, 1, n, f) != n) fail(PSC_E_IO, "write failed");
}

void read_all(FILE *f, void *p, size_t n) {
    if (n && fread(p, 1, n, f) != n) fail(PSC_E_FORMAT, "file truncated");
}

void write_section(FILE *f, uint32_t t, const void *data, size_t n) {
    SectionHeader sh{t, kCodecRaw, n, n, fnv1a(data, n)};
    std::vector<Bytef> z;
    const void *out = data;
    if (n >= kCompressAbove) {
        uLongf zn = compressBound((uLong)n);
        z.resize(zn);
        if (compress2(z.data(), &zn, static_cast<const Bytef *>(data), (uLong)n, Z_BEST_SPEED) != Z_OK)
            fail(PSC_E_IO, "compression failed");
        if (zn < n) {
            sh.codec = kCodecZlib;
            sh.stored_bytes = zn;
            out = z.data();
        }
    }
    write_all(f, &sh, sizeof sh);
    write_all(f, out, sh.stored_bytes);
}

template <class T>
void read_section(FILE *f, uint32_t t, std::vector<T> &dst) {
    SectionHeader sh;
    read_all(f, &sh, sizeof sh);
    if (sh.tag != t) fail(PSC_E_FORMAT, "unexpected section");
    if (sh.raw_bytes > kMaxSection || sh.stored_bytes > kMaxSection || sh.raw_bytes % sizeof(T))
        fail(PSC_E_FORMAT, "section size out of range");
    if (sh.codec != kCodecRaw && sh.codec != kCodecZlib) fail(PSC_E_FORMAT, "unknown section codec");
    dst.resize(sh.raw_bytes / sizeof(T));
    if (sh.codec == kCodecRaw) {
        if (sh.stored_bytes != sh.raw_bytes) fail(PSC_E_FORMAT, "section size mismatch");
        read_all(f, dst.data(), sh.raw_bytes);
    } else {
        std::vector<Bytef> z(sh.stored_bytes);
        read_all(f, z.data(), z.size());
        uLongf n = (uLongf)sh.raw_bytes;
        if (uncompress(reinterpret_cast<Bytef *>(dst.data()), &n, z.data(), (uLong)z.size()) != Z_OK ||
            n != sh.raw_bytes)
            fail(PSC_E_FORMAT, "corrupt compressed section");
    }
    if (fnv1a(dst.data(), sh.raw_bytes) != sh.checksum) fail(PSC_E_FORMAT, "section checksum mismatch");
}

// Everything the device kernels rely on, checked on a loaded handle;
// returns the number of skip edges.
int64_t check_loaded(const psc_handle &h) {
    auto bad = [](const std::string &m) { fail(PSC_E_FORMAT, "invalid classifier: " + m); };
    if (h.V <= 0 || h.W != (h.V + 31) / 32 || h.mask_stride < h.W || h.mask_stride % 64 || h.n_lex <= 0 ||
        h.n_lr <= 0 || h.n_classes <= 0)
        bad("sizes");
    if ((int64_t)h.masks.size() != (int64_t)h.n_classes * h.mask_stride) bad("mask table size");
    const int64_t T = (int64_t)h.table.size();
    if (h.rows_off != ((h.n_lex + 3) & ~3) || h.chains_off < h.rows_off || h.table_end < h.chains_off ||
        h.chains_off % 4 || h.table_end % 4 || T < h.table_end + kTablePad || T >= (int64_t)1 << 31)
        bad("table regions");
    const int32_t *t = h.table.data();
    // row and chain-entry starts, by kind
    std::vector<uint8_t> kind((size_t)T / 4, 0);   // 1 sparse, 2 dense, 3 chain entry
    for (int64_t pos = h.rows_off; pos < h.chains_off;) {
        const int32_t n = t[pos + 1];
        int64_t len = 0;
        if (n == -1) {
            kind[pos / 4] = 2;
            len = kRowHeader + 2 * (int64_t)h.n_lr;
        } else if (n >= 0 && n <= kSparseMax) {
            kind[pos / 4] = 1;
            len = kSparseHeader + kSparseEdge * (int64_t)n;
        } else {
            bad("row header");
        }
        pos += (len + 3) & ~3;
        if (pos > h.chains_off) bad("row crosses the chain region");
    }
    if (h.table_end > h.chains_off && h.n_lr > kMaxChainAlphabet) bad("chains with too large an alphabet");
    int run = 0;
    for (int64_t pos = h.chains_off; pos < h.table_end; pos += kChainEntry) {
        if ((t[pos] & 0xFFFF) == kSymJump) {
            if (run == 0) bad("empty chain");
            run = 0;
        } else {
            kind[pos / 4] = 3;
            if (++run > kChainMax) bad("chain longer than one wavefront load");
        }
    }
    if (run != 0) bad("chain without its jump entry");
    auto cls_ok = [&](int32_t c) { return c >= 0 && c < h.n_classes; };
    auto ref_ok = [&](int32_t r) {
        if (r < 0) return r >= -h.n_classes;
        const int64_t o = r & ~3;
        if (o >= T || o % 4) return false;
        const int k = r & 3;
        return (k == 0 && kind[o / 4] == 1) || (k == kRefDense && kind[o / 4] == 2) ||
               (k == kRefChain && kind[o / 4] == 3);
    };
    for (int32_t q = 0; q < h.n_lex; q++)
        if (!ref_ok(t[q])) bad("start ref");
    for (int64_t pos = h.rows_off; pos < h.chains_off;) {
        const int32_t *row = t + pos;
        if (!cls_ok(row[0])) bad("row end class");
        int64_t len = 0;
        if (row[1] == -1) {
            if (!ref_ok(row[2])) bad("dense row default");
            for (int32_t x = 0; x < h.n_lr; x++)
                if (!ref_ok(row[kRowHeader + 2 * x])) bad("dense row ref");
            len = kRowHeader + 2 * (int64_t)h.n_lr;
        } else {
            if (row[4] != kSymNone || !ref_ok(row[5])) bad("sparse row default");
            for (int32_t e = 0; e < row[1]; e++) {
                const int32_t *en = row + kSparseHeader + kSparseEdge * e;
                if (!ref_ok(en[1])) bad("sparse row ref");
                // in range and strictly increasing: the host walk searches them by bisection
                if (en[0] < 0 || en[0] >= h.n_lr || (e > 0 && en[0] <= en[-kSparseEdge])) bad("sparse row symbols");
            }
            len = kSparseHeader + kSparseEdge * (int64_t)row[1];
        }
        pos += (len + 3) & ~3;
    }
    for (int64_t pos = h.chains_off; pos < h.table_end; pos += kChainEntry) {
        const int32_t *e = t + pos;
        const uint32_t x = (uint32_t)e[0];
        if ((x & 0xFFFF) == kSymJump) {
            if (!ref_ok(e[2])) bad("chain jump ref");
            continue;
        }
        if (!cls_ok(e[3]) || !ref_ok(e[2]) || ((x >> 16) != kSymNone && !ref_ok(e[1]))) bad("chain entry refs");
    }
    // every skip is the one its ref's chain gives (so its target is a
    // validated jump ref)
    int64_t skips = 0;
    for (int64_t pos = h.rows_off; pos < h.chains_off;) {
        const int32_t *row = t + pos;
        int64_t len = kRowHeader + 2 * (int64_t)h.n_lr;
        if (row[1] == -1) {
            for (int32_t x = 0; x < h.n_lr; x++) {
                if (row[kRowHeader + 2 * x + 1] != chain_skip(t, T, row[kRowHeader + 2 * x])) bad("dense row skip");
                skips += row[kRowHeader + 2 * x + 1] != kNoSkip;
            }
        } else {
            if (row[6] != chain_skip(t, T, row[5])) bad("sparse row default skip");
            skips += row[6] != kNoSkip;
            for (int32_t e = 0; e < row[1]; e++) {
                const int32_t *en = row + kSparseHeader + kSparseEdge * e;
                if (en[2] != chain_skip(t, T, en[1])) bad("sparse row skip");
                skips += en[2] != kNoSkip;
            }
            len = kSparseHeader + kSparseEdge * (int64_t)row[1];
        }
        pos += (len + 3) & ~3;
    }
    // tail bits of every mask row are zero
    const uint32_t tail = h.V % 32 ? ~0u << (h.V % 32) : 0u;
    for (int32_t c = 0; c < h.n_classes; c++) {
        const uint32_t *m = h.masks.data() + (size_t)c * h.mask_stride;
        if (m[h.W - 1] & tail) bad("mask bits beyond the vocabulary");
        for (int32_t w = h.W; w < h.mask_stride; w++)
            if (m[w]) bad("mask row padding");
    }
    // the problem instance the device advance reads: its layout, then the
    // same checks psc_build applies to its inputs
    const AdvanceLayout &L = h.adv;
    const int64_t G = (int64_t)h.gram.size();
    if (L.n_term <= 0 || L.n_nt <= 0) bad("grammar sizes");
    const int64_t n_prod = L.prod_len - L.prod_lhs;
    if (L.lex_next != 0 || L.lex_accept != L.lex_next + (int64_t)h.n_lex * 256 ||
        L.ignored != L.lex_accept + h.n_lex || L.action != L.ignored + L.n_term ||
        L.go != L.action + (int64_t)h.n_lr * L.n_term || L.prod_lhs != L.go + (int64_t)h.n_lr * L.n_nt ||
        n_prod <= 0 || L.tok_off != L.prod_len + n_prod || G != L.tok_off + h.V + 1)
        bad("grammar layout");
    const int32_t *g = h.gram.data();
    std::vector<uint8_t> ign(L.n_term);
    for (int32_t i = 0; i < L.n_term; i++) {
        if (g[L.ignored + i] != 0 && g[L.ignored + i] != 1) bad("ignored flags");
        ign[i] = (uint8_t)g[L.ignored + i];
    }
    std::vector<int64_t> offs(h.V + 1);
    for (int32_t i = 0; i <= h.V; i++) offs[i] = g[L.tok_off + i];
    if (offs[h.V] != (int64_t)h.vbytes.size() && !(offs[h.V] == 0 && h.vbytes.size() == 1))
        bad("vocabulary bytes");
    psc_grammar pg{h.n_lex, g + L.lex_next, g + L.lex_accept, L.n_term, ign.data(), L.end_term, h.n_lr, L.n_nt,
                   g + L.action, g + L.go, (int32_t)n_prod, g + L.prod_lhs, g + L.prod_len};
    psc_vocab pv{h.V, h.vbytes.data(), offs.data(), L.eos};
    std::string msg;
    if (check_instance(&pg, &pv, &msg) != PSC_OK) bad(msg);
    return skips;
}

}  // namespace

extern "C" psc_status psc_save(const psc_handle *h, const char *path) {
    if (!h || !path) {
        set_error("psc_save: null argument");
        return PSC_E_INVALID_ARG;
    }
    try {
        File f;
        f.f = fopen(path, "wb");
        if (!f.f) fail(PSC_E_IO, std::string("cannot open ") + path);
        FileHeader fh{};
        std::memcpy(fh.magic, kMagic, 4);
        fh.version = kVersion;
        fh.header_bytes = sizeof(FileHeader);
        fh.n_sections = 4;
        fh.V = h->V;
        fh.W = h->W;
        fh.mask_stride = h->mask_stride;
        fh.n_lex = h->n_lex;
        fh.n_lr = h->n_lr;
        fh.n_classes = h->n_classes;
        fh.rows_off = h->rows_off;
        fh.chains_off = h->chains_off;
        fh.table_end = h->table_end;
        fh.info = h->info;
        fh.adv = h->adv;
        write_all(f.f, &fh, sizeof fh);
        write_section(f.f, tag("TABL"), h->table.data(), h->table.size() * sizeof(int32_t));
        write_section(f.f, tag("MASK"), h->masks.data(), h->masks.size() * sizeof(uint32_t));
        write_section(f.f, tag("GRAM"), h->gram.data(), h->gram.size() * sizeof(int32_t));
        write_section(f.f, tag("VBYT"), h->vbytes.data(), h->vbytes.size());
        if (fflush(f.f) != 0) fail(PSC_E_IO, "write failed");
        return PSC_OK;
    } catch (const StoreError &e) {
        set_error("psc_save: " + e.msg);
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("psc_save: out of host memory");
        return PSC_E_OOM;
    } catch (const std::exception &e) {
        set_error(std::string("psc_save: out of host resources (") + e.what() + ")");
        return PSC_E_OOM;
    }
}

extern "C" psc_status psc_load(const char *path, psc_handle **out) {
    if (!path || !out) {
        set_error("psc_load: null argument");
        return PSC_E_INVALID_ARG;
    }
    *out = nullptr;
    try {
        File f;
        f.f = fopen(path, "rb");
        if (!f.f) fail(PSC_E_IO, std::string("cannot open ") + path);
        FileHeader fh;
        read_all(f.f, &fh, sizeof fh);
        if (std::memcmp(fh.magic, kMagic, 4) != 0) fail(PSC_E_FORMAT, "not a classifier file");
        if (fh.version != kVersion || fh.header_bytes != sizeof(FileHeader) || fh.n_sections != 4)
            fail(PSC_E_FORMAT, "unsupported file version");
        std::unique_ptr<psc_handle> h(new psc_handle());
        h->V = fh.V;
        h->W = fh.W;
        h->mask_stride = fh.mask_stride;
        h->n_lex = fh.n_lex;
        h->n_lr = fh.n_lr;
        h->n_classes = fh.n_classes;
        h->rows_off = fh.rows_off;
        h->chains_off = fh.chains_off;
        h->table_end = fh.table_end;
        h->info = fh.info;
        h->adv = fh.adv;
        read_section(f.f, tag("TABL"), h->table);
        read_section(f.f, tag("MASK"), h->masks);
        read_section(f.f, tag("GRAM"), h->gram);
        read_section(f.f, tag("VBYT"), h->vbytes);
        const int64_t skips = check_loaded(*h);
        // the sizes the statistics report are the validated ones
        h->info.vocab_size = h->V;
        h->info.mask_words = h->W;
        h->info.mask_stride_words = h->mask_stride;
        h->info.n_lex_states = h->n_lex;
        h->info.n_lr_states = h->n_lr;
        h->info.n_classes = h->n_classes;
        h->info.table_bytes = (int64_t)h->table.size() * 4;
        h->info.mask_table_bytes = (int64_t)h->masks.size() * 4;
        h->info.skip_edges = skips;
        slice_masks(*h);
        h->info.device_bytes = (int64_t)h->device_bytes_needed();
        *out = h.release();
        return PSC_OK;
    } catch (const StoreError &e) {
        set_error("psc_load: " + e.msg);
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("psc_load: out of host memory");
        return PSC_E_OOM;
    } catch (const std::exception &e) {
        set_error(std::string("psc_load: out of host resources (") + e.what() + ")");
        return PSC_E_OOM;
    }
}
