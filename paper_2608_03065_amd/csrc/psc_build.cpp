// Offline construction of the parser-stack classifier (Algorithm 1).
//
// Input: the lexer T (byte DFA), the LR(1) tables realising the parser P,
// and the vocabulary V.  Output: one deterministic automaton over the stack
// alphabet (LR states) whose states carry precomputed token masks, flattened
// into int32 rows, plus a deduplicated table of mask rows.
//
// Route.  The paper builds, for every realizable terminal sequence w, the
// transducer P_w = P_eps o P~_w1 o P_eps o ... o P~_wn o P_eps (Sec. 3.3-3.4,
// eq. compose), drops its outputs (A_w), unions I_q A_w I_v over all q, v and
// w in R_q(v), then determinises and minimises (Sec. 3.5, eq. final_c).  We
// build the same language directly in determinised form: for one lexer
// state q at a time, a subset construction whose subset elements are the
// "threads" of those transducers, all run in lock step while the stack is
// read top-first:
//   * a thread stands for one terminal-sequence prefix (a node of the trie
//     of all sequences in R_q(V)) whose parser simulation has used up every
//     stack symbol it knows and is waiting for the next one;
//   * it waits either to skip k more symbols (a reduction popped below what
//     is known, P~/P_eps "readup") and then take the goto on nonterminal A
//     from the symbol after them, or -- the start thread -- for the top;
//   * reading a symbol resumes every thread: reductions run while the stack
//     they need is known (P_eps "execute"), a shift advances to the trie
//     child (P~_a), reaching a node that ends a sequence accepts that
//     sequence's tokens (the stack is stable right after a shift), and an
//     error drops the thread;
//   * a subset state is (set of waiting threads, mask of tokens accepted so
//     far); when the stack ends, waiting threads die and the state's mask is
//     its accepted set A_s (Sec. 3.5).
// Realizable sequences R_q(v) = x T_p (Sec. 3.1) come from lexing each token
// from q (longest match, one byte of lookahead), T_p being the terminals the
// pending lexeme can still become.  The automaton is then minimised (Moore),
// states whose class can no longer change are marked determined (walks stop
// there), and everything is flattened for the device.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <exception>
#include <memory>
#include <thread>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <sched.h>
#include <stdexcept>
#include <system_error>
#include <unordered_map>

#include "psc_internal.hpp"

namespace psc {

static thread_local std::string g_last_error;
void set_error(const std::string &msg) { g_last_error = msg; }

namespace {

struct BuildError : std::runtime_error {
    psc_status code;
    BuildError(psc_status c, const std::string &m) : std::runtime_error(m), code(c) {}
};

inline uint64_t mix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// Interning of variable-length keys (open addressing over ids).
template <class T>
class Interner {
  public:
    int32_t find_or_add(const T *key, size_t n, bool *added) {
        uint64_t h = hash(key, n);
        if ((ids_.size() + 1) * 2 > slots_.size()) grow();
        size_t mask = slots_.size() - 1;
        size_t i = h & mask;
        while (true) {
            int32_t id = slots_[i];
            if (id < 0) break;
            if (hashes_[id] == h && len(id) == n && std::equal(key, key + n, data(id))) {
                *added = false;
                return id;
            }
            i = (i + 1) & mask;
        }
        int32_t id = (int32_t)ids_.size();
        slots_[i] = id;
        ids_.push_back(pool_.size());
        hashes_.push_back(h);
        pool_.insert(pool_.end(), key, key + n);
        ends_.push_back(pool_.size());
        *added = true;
        return id;
    }
    size_t size() const { return ids_.size(); }
    const T *data(int32_t id) const { return pool_.data() + ids_[id]; }
    size_t len(int32_t id) const { return ends_[id] - ids_[id]; }
    void clear() {
        pool_.clear(); ids_.clear(); ends_.clear(); hashes_.clear();
        slots_.assign(16, -1);
        pool_.shrink_to_fit(); ids_.shrink_to_fit(); ends_.shrink_to_fit(); hashes_.shrink_to_fit();
    }
    Interner() { slots_.assign(16, -1); }

  private:
    static uint64_t hash(const T *k, size_t n) {
        uint64_t h = 0x1234567ull + n;
        for (size_t i = 0; i < n; i++) h = mix64(h ^ (uint64_t)k[i]);
        return h;
    }
    void grow() {
        std::vector<int32_t> ns(slots_.size() * 2, -1);
        size_t mask = ns.size() - 1;
        for (size_t id = 0; id < ids_.size(); id++) {
            size_t i = hashes_[id] & mask;
            while (ns[i] >= 0) i = (i + 1) & mask;
            ns[i] = (int32_t)id;
        }
        slots_.swap(ns);
    }
    std::vector<T> pool_;
    std::vector<size_t> ids_, ends_;
    std::vector<uint64_t> hashes_;
    std::vector<int32_t> slots_;
};

// ------------------------------------------------------------------ grammar

struct Gram {
    int32_t nQ, nT, nPi, nN, nP, endT;
    const int32_t *lex_next, *lex_accept, *action, *go, *plhs, *plen;
    const uint8_t *ign;
    int32_t act(int32_t s, int32_t t) const { return action[(int64_t)s * nT + t]; }
    int32_t gto(int32_t s, int32_t A) const { return go[(int64_t)s * nN + A]; }
};

void validate(const psc_grammar *g, const psc_vocab *v) {
    auto bad = [](const std::string &m) { throw BuildError(PSC_E_GRAMMAR, m); };
    if (g->n_lex_states <= 0 || g->n_terminals <= 0 || g->n_lr_states <= 0 ||
        g->n_nonterminals <= 0 || g->n_productions <= 0)
        throw BuildError(PSC_E_INVALID_ARG, "grammar sizes must be positive");
    if (!g->lex_next || !g->lex_accept || !g->terminal_ignored || !g->action || !g->goto_table ||
        !g->prod_lhs || !g->prod_len)
        throw BuildError(PSC_E_INVALID_ARG, "null grammar array");
    if (g->n_nonterminals >= 32767 || g->n_lr_states >= (1 << 29))
        throw BuildError(PSC_E_LIMIT, "grammar too large for the table encoding");
    if (g->end_terminal < 0 || g->end_terminal >= g->n_terminals) bad("end_terminal out of range");
    if (g->lex_accept[0] != -1) bad("lexer state 0 (q0) must not be accepting");
    for (int64_t i = 0; i < (int64_t)g->n_lex_states * 256; i++) {
        int32_t x = g->lex_next[i];
        if (x < -1 || x >= g->n_lex_states) bad("lexer transition out of range");
        if (x == 0) bad("no lexer transition may lead back to q0");
    }
    for (int32_t i = 0; i < g->n_lex_states; i++)
        if (g->lex_accept[i] < -1 || g->lex_accept[i] >= g->n_terminals ||
            g->lex_accept[i] == g->end_terminal)
            bad("lexer accept label out of range");
    for (int32_t p = 0; p < g->n_productions; p++)
        if (g->prod_lhs[p] < 0 || g->prod_lhs[p] >= g->n_nonterminals || g->prod_len[p] < 0)
            bad("production out of range");
    for (int64_t i = 0; i < (int64_t)g->n_lr_states * g->n_terminals; i++) {
        int32_t a = g->action[i];
        int k = a & 3;
        if (k == 1 && ((a >> 2) < 0 || (a >> 2) >= g->n_lr_states)) bad("shift target out of range");
        if (k == 2 && ((a >> 2) < 0 || (a >> 2) >= g->n_productions)) bad("reduce production out of range");
        if (k == 0 && a != 0) bad("error entries must be 0");
    }
    for (int64_t i = 0; i < (int64_t)g->n_lr_states * g->n_nonterminals; i++)
        if (g->goto_table[i] < -1 || g->goto_table[i] >= g->n_lr_states) bad("goto out of range");
    if (v->n_tokens <= 0 || !v->offsets || (!v->bytes && v->offsets[v->n_tokens] > 0))
        throw BuildError(PSC_E_INVALID_ARG, "empty or null vocabulary");
    if (v->eos_id < -1 || v->eos_id >= v->n_tokens) throw BuildError(PSC_E_INVALID_ARG, "eos_id out of range");
    if (v->offsets[0] != 0) bad("vocabulary offsets must start at 0");
    for (int32_t t = 0; t < v->n_tokens; t++) {
        int64_t n = v->offsets[t + 1] - v->offsets[t];
        if (n < 0) bad("vocabulary offsets must be non-decreasing");
        if (n == 0 && t != v->eos_id) bad("only the EOS token may have an empty spelling");
        if (n > 0 && t == v->eos_id) bad("the EOS token must have an empty spelling");
    }
}

// T_p for every lexer state p (Sec. 3.1): the terminals whose accepting
// states are reachable from p, and whether "nothing more" is possible
// (p == q0, or an ignored terminal is reachable).
struct Completions {
    std::vector<std::vector<int32_t>> terms;  // non-ignored terminals per p
    std::vector<uint8_t> eps;
};

Completions completions(const Gram &G) {
    int32_t words = (G.nT + 63) / 64;
    std::vector<uint64_t> R((size_t)G.nQ * words, 0);
    std::vector<std::vector<int32_t>> succ(G.nQ);
    for (int32_t p = 0; p < G.nQ; p++) {
        if (G.lex_accept[p] >= 0) R[(size_t)p * words + G.lex_accept[p] / 64] |= 1ull << (G.lex_accept[p] % 64);
        for (int c = 0; c < 256; c++) {
            int32_t r = G.lex_next[(int64_t)p * 256 + c];
            if (r >= 0 && r != p) succ[p].push_back(r);
        }
        std::sort(succ[p].begin(), succ[p].end());
        succ[p].erase(std::unique(succ[p].begin(), succ[p].end()), succ[p].end());
    }
    bool changed = true;
    while (changed) {
        changed = false;
        for (int32_t p = G.nQ - 1; p >= 0; p--) {
            uint64_t *rp = &R[(size_t)p * words];
            for (int32_t r : succ[p]) {
                const uint64_t *rr = &R[(size_t)r * words];
                for (int32_t k = 0; k < words; k++) {
                    uint64_t nv = rp[k] | rr[k];
                    if (nv != rp[k]) { rp[k] = nv; changed = true; }
                }
            }
        }
    }
    Completions C;
    C.terms.resize(G.nQ);
    C.eps.assign(G.nQ, 0);
    for (int32_t p = 0; p < G.nQ; p++) {
        if (p == 0) C.eps[p] = 1;
        for (int32_t t = 0; t < G.nT; t++) {
            if (!(R[(size_t)p * words + t / 64] >> (t % 64) & 1)) continue;
            if (G.ign[t]) C.eps[p] = 1;
            else C.terms[p].push_back(t);
        }
    }
    return C;
}

// ------------------------------------------------------- vocabulary trie

struct VocabTrie {
    std::vector<int32_t> depth, subtree_end, tok_begin, tok_end;
    std::vector<uint8_t> byte;
    std::vector<int32_t> toks;   // token ids ending at nodes, grouped by node
};

VocabTrie vocab_trie(const psc_vocab *v) {
    std::vector<int32_t> ids;
    for (int32_t t = 0; t < v->n_tokens; t++)
        if (t != v->eos_id) ids.push_back(t);
    auto spell = [&](int32_t t) {
        return std::pair<const uint8_t *, int64_t>(v->bytes + v->offsets[t], v->offsets[t + 1] - v->offsets[t]);
    };
    std::sort(ids.begin(), ids.end(), [&](int32_t a, int32_t b) {
        auto [pa, na] = spell(a);
        auto [pb, nb] = spell(b);
        int c = std::memcmp(pa, pb, (size_t)std::min(na, nb));
        return c != 0 ? c < 0 : (na != nb ? na < nb : a < b);
    });
    VocabTrie T;
    T.depth.push_back(0);
    T.byte.push_back(0);
    std::vector<int32_t> node_tok_owner;  // node id per entry of toks (built in node order)
    std::vector<std::pair<int32_t, int32_t>> ends;  // (node, token)
    std::vector<int32_t> path{0};  // node at each depth of the previous token
    const uint8_t *prev = nullptr;
    int64_t prev_n = 0;
    for (int32_t t : ids) {
        auto [p, n] = spell(t);
        int64_t lcp = 0;
        if (prev) while (lcp < n && lcp < prev_n && p[lcp] == prev[lcp]) lcp++;
        path.resize((size_t)lcp + 1);
        for (int64_t d = lcp; d < n; d++) {
            T.depth.push_back((int32_t)d + 1);
            T.byte.push_back(p[d]);
            path.push_back((int32_t)T.depth.size() - 1);
        }
        ends.emplace_back(path[(size_t)n], t);
        prev = p;
        prev_n = n;
    }
    int32_t N = (int32_t)T.depth.size();
    std::sort(ends.begin(), ends.end());
    T.tok_begin.assign(N, 0);
    T.tok_end.assign(N, 0);
    size_t e = 0;
    for (int32_t i = 0; i < N; i++) {
        T.tok_begin[i] = (int32_t)T.toks.size();
        while (e < ends.size() && ends[e].first == i) T.toks.push_back(ends[e++].second);
        T.tok_end[i] = (int32_t)T.toks.size();
    }
    T.subtree_end.assign(N, N);
    std::vector<int32_t> open;
    for (int32_t i = 0; i < N; i++) {
        while (!open.empty() && T.depth[open.back()] >= T.depth[i]) {
            T.subtree_end[open.back()] = i;
            open.pop_back();
        }
        open.push_back(i);
    }
    return T;
}

// ----------------------------------------------------------- automaton

constexpr int32_t kInitA = 0xFFFF;   // "read the top" thread marker

inline uint64_t pack_thread(int32_t node, int32_t k, int32_t A) {
    return ((uint64_t)(uint32_t)node << 32) | ((uint64_t)(uint32_t)k << 16) | (uint64_t)(uint32_t)A;
}
inline int32_t th_node(uint64_t t) { return (int32_t)(t >> 32); }
inline int32_t th_k(uint64_t t) { return (int32_t)((t >> 16) & 0xFFFF); }
inline int32_t th_A(uint64_t t) { return (int32_t)(t & 0xFFFF); }

// Moore refinement over total transition functions (default + explicit
// edges).  States start in blocks of equal `label`; returns the block of
// every state (ids 0..*n_blocks-1).
std::vector<int32_t> moore(int32_t N, const std::vector<int32_t> &label, const std::vector<int32_t> &def,
                           const std::vector<int32_t> &ebeg, const std::vector<int32_t> &eend,
                           const std::vector<int32_t> &esym, const std::vector<int32_t> &etgt,
                           int32_t *n_blocks_out) {
    std::vector<int32_t> block(N);
    int32_t nb;
    {
        Interner<int32_t> in;
        bool a;
        for (int32_t s = 0; s < N; s++) block[s] = in.find_or_add(&label[s], 1, &a);
        nb = (int32_t)in.size();
    }
    std::vector<int32_t> sig, nbk(N);
    while (true) {
        Interner<int32_t> in;
        for (int32_t s = 0; s < N; s++) {
            sig.clear();
            int32_t db = block[def[s]];
            sig.push_back(block[s]);
            sig.push_back(db);
            for (int32_t e = ebeg[s]; e < eend[s]; e++) {
                int32_t tb = block[etgt[e]];
                if (tb != db) { sig.push_back(esym[e]); sig.push_back(tb); }
            }
            bool a;
            nbk[s] = in.find_or_add(sig.data(), sig.size(), &a);
        }
        int32_t nnb = (int32_t)in.size();
        block.swap(nbk);
        if (nnb == nb) break;
        nb = nnb;
    }
    *n_blocks_out = nb;
    return block;
}

// The stack known to a running simulation (top at the back); bounded by the
// longest realizable terminal sequence plus the pushes of its reductions.
constexpr int32_t kMaxBeta = 192;
struct Beta {
    int32_t n = 0;
    int32_t s[kMaxBeta];
    void push(int32_t v) {
        if (n >= kMaxBeta) throw BuildError(PSC_E_LIMIT, "simulated stack exceeds 192 symbols");
        s[n++] = v;
    }
    int32_t top() const { return s[n - 1]; }
};

// One builder per thread; it processes lexer states one at a time and
// appends each one's minimised sub-automaton to its output arrays.
struct Builder {
    const Gram &G;
    const psc_vocab *vocab;
    const Completions &C;
    const VocabTrie &VT;
    int32_t V, W;
    bool verbose;

    // outputs: mask classes (class 0 = all zero) and automaton states
    Interner<uint32_t> masks;
    std::vector<int32_t> st_cls, st_def, st_ebeg, st_eend;
    std::vector<int32_t> e_sym, e_tgt;
    std::vector<int32_t> start_state;   // per lexer state
    std::vector<std::vector<int32_t>> goto_sources;  // per nonterminal
    int64_t states_built = 0;
    std::atomic<int64_t> *total_states = nullptr;
    int64_t max_states = 1'000'000'000;   // built over all lexer states; PSC_BUILD_MAX_STATES overrides

    // per-q: trie of realizable terminal sequences
    std::vector<int32_t> tn_label, tn_child_beg, tn_child_end, tn_children, tn_grp_beg, tn_grp_end, tn_grps;
    std::vector<std::vector<int32_t>> grp_tokens;
    std::vector<uint64_t> node_ka, node_kb;        // random keys of trie nodes

    // per-q: subset states.  A state is (waiting threads, accepted trie
    // nodes); the accepted set is identified by a 128-bit order-independent
    // hash (XOR of node keys -- a node is accepted at most once along a
    // walk) and reconstructed, when needed, from the breadth-first tree:
    // each state keeps its parent and the nodes accepted on that edge.
    Interner<uint64_t> qstates;                     // key: [acc_a, acc_b, threads...]
    std::vector<int32_t> qs_parent, qs_dbeg, qs_dend, delta_pool;
    std::vector<uint64_t> qs_acca, qs_accb;
    std::vector<int32_t> qs_def, qs_ebeg, qs_eend, qe_sym, qe_tgt;

    // per-q: resumption memo (trie node, symbol, nonterminal) -> results
    std::unordered_map<uint64_t, int32_t> memo;
    std::vector<int32_t> memo_wb, memo_we, memo_ab, memo_ae, memo_a;
    std::vector<uint64_t> memo_w;

    std::vector<uint64_t> newW;
    std::vector<int32_t> acc;

    // Valid stacks only: the symbol below X on a parser stack is an LR
    // predecessor of X (it has a shift or goto into X), and the top is a
    // shift target or the start state.  Each subset state carries the set of
    // symbols that can come next on a valid stack (an interned bitset over
    // Pi) and only those transitions are expanded; any other symbol belongs
    // to no valid stack and falls to the default.
    int32_t pw;                                       // uint64 words per symbol set
    std::vector<uint64_t> pred_bits;                  // [nPi][pw]
    std::vector<uint64_t> tops_bits;                  // [pw]
    Interner<uint64_t> symsets;
    std::vector<uint64_t> setbuf;

    Builder(const Gram &g, const psc_vocab *v, const Completions &c, const VocabTrie &vt, bool verb)
        : G(g), vocab(v), C(c), VT(vt), V(v->n_tokens), W((v->n_tokens + 31) / 32), verbose(verb) {
        std::vector<uint32_t> zero(W, 0);
        bool added;
        masks.find_or_add(zero.data(), W, &added);
        goto_sources.resize(G.nN);
        for (int32_t s = 0; s < G.nPi; s++)
            for (int32_t A = 0; A < G.nN; A++)
                if (G.gto(s, A) >= 0) goto_sources[A].push_back(s);
        pw = (G.nPi + 63) / 64;
        pred_bits.assign((size_t)G.nPi * pw, 0);
        tops_bits.assign(pw, 0);
        tops_bits[0] |= 1;
        for (int32_t s = 0; s < G.nPi; s++) {
            for (int32_t t = 0; t < G.nT; t++) {
                int32_t a = G.act(s, t);
                if ((a & 3) == 1) {
                    int32_t x = a >> 2;
                    pred_bits[(size_t)x * pw + s / 64] |= 1ull << (s % 64);
                    tops_bits[x / 64] |= 1ull << (x % 64);
                }
            }
            for (int32_t A = 0; A < G.nN; A++) {
                int32_t x = G.gto(s, A);
                if (x >= 0) pred_bits[(size_t)x * pw + s / 64] |= 1ull << (s % 64);
            }
        }
        setbuf.resize(pw);
    }

    int32_t symset_id(const uint64_t *bits) {
        bool a;
        return symsets.find_or_add(bits, pw, &a);
    }
    bool in_set(int32_t set, int32_t X) const { return (symsets.data(set)[X / 64] >> (X % 64)) & 1; }

    // ---- lexical pass for one q: group tokens by (emitted x, end state p)
    void lexical_pass(int32_t q, Interner<int32_t> &groups) {
        int32_t N = (int32_t)VT.depth.size();
        int32_t maxd = 0;
        for (int32_t d : VT.depth) maxd = std::max(maxd, d);
        std::vector<int32_t> cur(maxd + 2), emlen(maxd + 2), embuf(maxd + 2), key(maxd + 3);
        cur[0] = q;
        emlen[0] = 0;
        grp_tokens.clear();
        int32_t i = 1;
        while (i < N) {
            int32_t d = VT.depth[i];
            uint8_t c = VT.byte[i];
            int32_t s = cur[d - 1];
            int32_t em = emlen[d - 1];
            int32_t nx = G.lex_next[(int64_t)s * 256 + c];
            if (nx < 0) {
                int32_t t = (s != 0) ? G.lex_accept[s] : -1;
                if (t >= 0) {
                    if (!G.ign[t]) embuf[em++] = t;
                    nx = G.lex_next[c];
                }
            }
            if (nx < 0) {           // the lexer dies: no token below this node is valid
                i = VT.subtree_end[i];
                continue;
            }
            cur[d] = nx;
            emlen[d] = em;
            if (VT.tok_end[i] > VT.tok_begin[i]) {
                key[0] = nx;
                for (int32_t k = 0; k < em; k++) key[1 + k] = embuf[k];
                bool added;
                int32_t gid = groups.find_or_add(key.data(), (size_t)em + 1, &added);
                if (added) grp_tokens.emplace_back();
                auto &lst = grp_tokens[gid];
                lst.insert(lst.end(), VT.toks.begin() + VT.tok_begin[i], VT.toks.begin() + VT.tok_end[i]);
            }
            i++;
        }
    }

    // ---- the trie of realizable terminal sequences R_q(V) for one q
    void sequence_trie(int32_t q, const Interner<int32_t> &groups) {
        std::vector<int32_t> label{-1};
        std::unordered_map<uint64_t, int32_t> kid;
        std::vector<std::pair<int32_t, int32_t>> node_grp;   // (node, group)
        auto child = [&](int32_t n, int32_t t) {
            uint64_t k = ((uint64_t)(uint32_t)n << 32) | (uint32_t)t;
            auto it = kid.find(k);
            if (it != kid.end()) return it->second;
            int32_t id = (int32_t)label.size();
            label.push_back(t);
            kid.emplace(k, id);
            return id;
        };
        int32_t n_groups = (int32_t)groups.size();
        for (int32_t g = 0; g < n_groups; g++) {
            const int32_t *k = groups.data(g);
            size_t len = groups.len(g);
            int32_t p = k[0];
            int32_t n = 0;
            for (size_t j = 1; j < len; j++) n = child(n, k[j]);
            if (C.eps[p]) node_grp.emplace_back(n, g);
            for (int32_t t : C.terms[p]) node_grp.emplace_back(child(n, t), g);
        }
        // EOS: the pending lexeme must end here, then $end must be accepted
        if (vocab->eos_id >= 0) {
            int32_t n = -1;
            if (q == 0) n = child(0, G.endT);
            else if (G.lex_accept[q] >= 0) {
                int32_t t = G.lex_accept[q];
                n = G.ign[t] ? child(0, G.endT) : child(child(0, t), G.endT);
            }
            if (n >= 0) {
                grp_tokens.push_back({vocab->eos_id});
                node_grp.emplace_back(n, (int32_t)grp_tokens.size() - 1);
            }
        }
        int32_t N = (int32_t)label.size();
        tn_label = label;
        // children sorted by terminal, CSR
        std::vector<std::pair<uint64_t, int32_t>> edges(kid.begin(), kid.end());
        std::sort(edges.begin(), edges.end(), [&](const auto &a, const auto &b) {
            uint32_t pa = (uint32_t)(a.first >> 32), pb = (uint32_t)(b.first >> 32);
            return pa != pb ? pa < pb : (uint32_t)a.first < (uint32_t)b.first;
        });
        tn_child_beg.assign(N, 0);
        tn_child_end.assign(N, 0);
        tn_children.clear();
        for (auto &e : edges) {
            int32_t par = (int32_t)(e.first >> 32);
            if (tn_child_end[par] == tn_child_beg[par]) tn_child_beg[par] = (int32_t)tn_children.size();
            tn_children.push_back(e.second);
            tn_child_end[par] = (int32_t)tn_children.size();
        }
        std::sort(node_grp.begin(), node_grp.end());
        tn_grp_beg.assign(N, 0);
        tn_grp_end.assign(N, 0);
        tn_grps.clear();
        for (auto &ng : node_grp) {
            if (tn_grp_end[ng.first] == tn_grp_beg[ng.first]) tn_grp_beg[ng.first] = (int32_t)tn_grps.size();
            tn_grps.push_back(ng.second);
            tn_grp_end[ng.first] = (int32_t)tn_grps.size();
        }
        node_ka.resize(N);
        node_kb.resize(N);
        for (int32_t n = 0; n < N; n++) {
            uint64_t base = ((uint64_t)(uint32_t)q << 32) | (uint32_t)n;
            node_ka[n] = mix64(base ^ 0x5A17C0DEull);
            node_kb[n] = mix64(base * 0x9E3779B97F4A7C15ull + 0x1234ull);
        }
    }

    // ---- parser simulation on a known stack top (beta, top at the back)
    void run(int32_t c, Beta &beta) {
        const int32_t t = tn_label[c];
        for (;;) {
            int32_t a = G.act(beta.top(), t);
            switch (a & 3) {
            case 1:                       // shift: the stack is stable again
                beta.push(a >> 2);
                visit(c, beta);
                return;
            case 3:                       // accept ($end)
                acc.push_back(c);
                return;
            case 2: {                     // reduce
                int32_t p = a >> 2, m = G.plen[p], A = G.plhs[p];
                if (m < beta.n) {
                    beta.n -= m;
                    int32_t g = G.gto(beta.top(), A);
                    if (g < 0) return;
                    beta.push(g);
                    continue;
                }
                int32_t k = m - beta.n;
                if (k > 0xFFFE) throw BuildError(PSC_E_LIMIT, "production too long");
                newW.push_back(pack_thread(c, k, A));
                return;
            }
            default:
                return;
            }
        }
    }

    void visit(int32_t c, const Beta &beta) {
        if (tn_grp_end[c] > tn_grp_beg[c]) acc.push_back(c);
        for (int32_t j = tn_child_beg[c]; j < tn_child_end[c]; j++) {
            Beta b2;
            b2.n = beta.n;
            std::memcpy(b2.s, beta.s, sizeof(int32_t) * beta.n);
            run(tn_children[j], b2);
        }
    }

    // resume a thread waiting for its goto base X (memoised)
    void resume(int32_t c, int32_t X, int32_t A) {
        const uint64_t key = (uint64_t)(uint32_t)c * ((uint64_t)G.nPi * 32768ull) + (uint64_t)X * 32768ull + (uint64_t)A;
        auto it = memo.find(key);
        if (it == memo.end()) {
            size_t w0 = newW.size(), a0 = acc.size();
            int32_t g = G.gto(X, A);
            if (g >= 0) {
                Beta beta;
                beta.n = 0;
                beta.push(X);
                beta.push(g);
                run(c, beta);
            }
            int32_t id = (int32_t)memo_wb.size();
            memo_wb.push_back((int32_t)memo_w.size());
            memo_w.insert(memo_w.end(), newW.begin() + w0, newW.end());
            memo_we.push_back((int32_t)memo_w.size());
            memo_ab.push_back((int32_t)memo_a.size());
            memo_a.insert(memo_a.end(), acc.begin() + a0, acc.end());
            memo_ae.push_back((int32_t)memo_a.size());
            memo.emplace(key, id);
            return;
        }
        int32_t id = it->second;
        newW.insert(newW.end(), memo_w.begin() + memo_wb[id], memo_w.begin() + memo_we[id]);
        acc.insert(acc.end(), memo_a.begin() + memo_ab[id], memo_a.begin() + memo_ae[id]);
    }

    // state id for (threads, accepted set); queue new ones
    int32_t intern(std::vector<uint64_t> &th, uint64_t acca, uint64_t accb, int32_t next_set, int32_t parent,
                   const std::vector<int32_t> &delta, std::vector<int32_t> &queue) {
        std::sort(th.begin(), th.end());
        th.erase(std::unique(th.begin(), th.end()), th.end());
        std::vector<uint64_t> key;
        key.reserve(th.size() + 3);
        key.push_back(acca);
        key.push_back(accb);
        key.push_back((uint64_t)(uint32_t)next_set);
        key.insert(key.end(), th.begin(), th.end());
        bool added;
        int32_t id = qstates.find_or_add(key.data(), key.size(), &added);
        if (added) {
            qs_parent.push_back(parent);
            qs_dbeg.push_back((int32_t)delta_pool.size());
            delta_pool.insert(delta_pool.end(), delta.begin(), delta.end());
            qs_dend.push_back((int32_t)delta_pool.size());
            qs_acca.push_back(acca);
            qs_accb.push_back(accb);
            qs_def.push_back(id);
            qs_ebeg.push_back(0);
            qs_eend.push_back(0);
            queue.push_back(id);
            states_built++;
            if (total_states && total_states->fetch_add(1) + 1 > max_states)
                throw BuildError(PSC_E_LIMIT, "automaton exceeds " + std::to_string(max_states) +
                                                  " states (PSC_BUILD_MAX_STATES)");
        }
        return id;
    }

    int32_t step(int32_t sid, const uint64_t *th, size_t n, uint64_t acca, uint64_t accb, int32_t X,
                 std::vector<int32_t> &queue) {
        newW.clear();
        acc.clear();
        for (size_t i = 0; i < n; i++) {
            uint64_t t = th[i];
            int32_t c = th_node(t), k = th_k(t), A = th_A(t);
            if (A == kInitA) {
                for (int32_t j = tn_child_beg[c]; j < tn_child_end[c]; j++) {
                    Beta beta;
                    beta.n = 0;
                    beta.push(X);
                    run(tn_children[j], beta);
                }
            } else if (k > 0) {
                newW.push_back(pack_thread(c, k - 1, A));
            } else {
                resume(c, X, A);
            }
        }
        std::sort(acc.begin(), acc.end());
        acc.erase(std::unique(acc.begin(), acc.end()), acc.end());
        for (int32_t c : acc) {
            acca ^= node_ka[c];
            accb ^= node_kb[c];
        }
        std::vector<uint64_t> w2 = newW;
        return intern(w2, acca, accb, symset_id(&pred_bits[(size_t)X * pw]), sid, acc, queue);
    }

    // mask of the tokens accepted on the breadth-first path to state s
    int32_t class_of(int32_t s, std::vector<uint32_t> &row) {
        std::fill(row.begin(), row.end(), 0u);
        for (int32_t x = s; x >= 0; x = qs_parent[x])
            for (int32_t d = qs_dbeg[x]; d < qs_dend[x]; d++) {
                int32_t c = delta_pool[d];
                for (int32_t j = tn_grp_beg[c]; j < tn_grp_end[c]; j++)
                    for (int32_t tok : grp_tokens[tn_grps[j]]) row[tok >> 5] |= 1u << (tok & 31);
            }
        bool added;
        return masks.find_or_add(row.data(), W, &added);
    }

    void clear_q() {
        qstates.clear();
        qs_parent.clear(); qs_dbeg.clear(); qs_dend.clear(); delta_pool.clear();
        qs_acca.clear(); qs_accb.clear(); qs_def.clear(); qs_ebeg.clear(); qs_eend.clear();
        qe_sym.clear(); qe_tgt.clear();
        memo.clear(); memo_wb.clear(); memo_we.clear(); memo_ab.clear(); memo_ae.clear();
        memo_a.clear(); memo_w.clear();
        for (auto *v : {&qs_parent, &qs_dbeg, &qs_dend, &delta_pool, &qs_def, &qs_ebeg, &qs_eend, &qe_sym, &qe_tgt,
                        &memo_wb, &memo_we, &memo_ab, &memo_ae, &memo_a})
            v->shrink_to_fit();
        qs_acca.shrink_to_fit(); qs_accb.shrink_to_fit(); memo_w.shrink_to_fit();
        std::unordered_map<uint64_t, int32_t>().swap(memo);
    }

    void build_for_lexer_state(int32_t q) {
        auto t_start = std::chrono::steady_clock::now();
        Interner<int32_t> groups;
        lexical_pass(q, groups);
        sequence_trie(q, groups);
        clear_q();
        std::vector<int32_t> queue;
        // the root's groups (sequence x = nothing more) are accepted at once
        std::vector<int32_t> root_acc;
        uint64_t a0 = 0, b0 = 0;
        if (tn_grp_end[0] > tn_grp_beg[0]) {
            root_acc.push_back(0);
            a0 ^= node_ka[0];
            b0 ^= node_kb[0];
        }
        std::vector<uint64_t> init{pack_thread(0, 0, kInitA)};
        int32_t start = intern(init, a0, b0, symset_id(tops_bits.data()), -1, root_acc, queue);
        std::vector<uint64_t> key, dW;
        std::vector<int32_t> syms, none;
        std::vector<uint8_t> seen(G.nPi, 0);
        auto t_last = t_start;
        size_t max_threads = 0;
        for (size_t qi = 0; qi < queue.size(); qi++) {
            if (verbose) {
                auto now = std::chrono::steady_clock::now();
                if (std::chrono::duration<double>(now - t_last).count() > 5.0) {
                    t_last = now;
                    std::fprintf(stderr, "psc_build:   q=%d %.0fs states %zu/%zu max-threads %zu memo %zu\n", q,
                                 std::chrono::duration<double>(now - t_start).count(), qi, queue.size(),
                                 max_threads, memo.size());
                }
            }
            int32_t sid = queue[qi];
            key.assign(qstates.data(sid), qstates.data(sid) + qstates.len(sid));
            uint64_t acca = key[0], accb = key[1];
            const int32_t next_set = (int32_t)key[2];
            const uint64_t *th = key.data() + 3;
            size_t n = key.size() - 3;
            max_threads = std::max(max_threads, n);
            // default transition: waiting-to-skip threads advance, others die
            dW.clear();
            bool init_thread = false;
            syms.clear();
            for (size_t i = 0; i < n; i++) {
                int32_t k = th_k(th[i]), A = th_A(th[i]);
                if (A == kInitA) init_thread = true;
                else if (k > 0) dW.push_back(pack_thread(th_node(th[i]), k - 1, A));
                else
                    for (int32_t X : goto_sources[A])
                        if (!seen[X] && in_set(next_set, X)) { seen[X] = 1; syms.push_back(X); }
            }
            for (int32_t X : syms) seen[X] = 0;
            if (init_thread) {
                syms.clear();
                for (int32_t X = 0; X < G.nPi; X++)
                    if (in_set(next_set, X)) syms.push_back(X);
            }
            std::sort(syms.begin(), syms.end());
            // the symbols that take the default: valid next symbols not in syms
            std::fill(setbuf.begin(), setbuf.end(), 0ull);
            {
                const uint64_t *ns = symsets.data(next_set);
                size_t j = 0;
                for (int32_t w = 0; w < pw; w++) {
                    uint64_t m = ns[w];
                    while (m) {
                        int32_t X = w * 64 + __builtin_ctzll(m);
                        m &= m - 1;
                        while (j < syms.size() && syms[j] < X) j++;
                        if (j < syms.size() && syms[j] == X) continue;
                        const uint64_t *pb = &pred_bits[(size_t)X * pw];
                        for (int32_t k = 0; k < pw; k++) setbuf[k] |= pb[k];
                    }
                }
            }
            int32_t def = n == 0 ? sid : intern(dW, acca, accb, symset_id(setbuf.data()), sid, none, queue);
            int32_t ebeg = (int32_t)qe_sym.size();
            for (int32_t X : syms) {
                int32_t tgt = step(sid, th, n, acca, accb, X, queue);
                if (tgt != def) {
                    qe_sym.push_back(X);
                    qe_tgt.push_back(tgt);
                }
            }
            qs_def[sid] = def;
            qs_ebeg[sid] = ebeg;
            qs_eend[sid] = (int32_t)qe_sym.size();
        }
        // minimise this lexer state's automaton (accepted-set hashes as the
        // initial partition), then compute the mask of each block once
        int32_t N = (int32_t)queue.size();
        std::vector<int32_t> label(N);
        {
            Interner<uint64_t> in;
            bool a;
            for (int32_t s = 0; s < N; s++) {
                uint64_t k2[2] = {qs_acca[s], qs_accb[s]};
                label[s] = in.find_or_add(k2, 2, &a);
            }
        }
        int32_t nb = 0;
        std::vector<int32_t> block = moore(N, label, qs_def, qs_ebeg, qs_eend, qe_sym, qe_tgt, &nb);
        std::vector<int32_t> rep(nb, -1);
        for (int32_t s = 0; s < N; s++)
            if (rep[block[s]] < 0) rep[block[s]] = s;
        std::vector<uint32_t> row(W);
        int32_t off = (int32_t)st_cls.size();
        for (int32_t b = 0; b < nb; b++) {
            int32_t s = rep[b];
            st_cls.push_back(class_of(s, row));
            int32_t db = block[qs_def[s]];
            st_def.push_back(off + db);
            st_ebeg.push_back((int32_t)e_sym.size());
            for (int32_t e = qs_ebeg[s]; e < qs_eend[s]; e++) {
                int32_t tb = block[qe_tgt[e]];
                if (tb != db) { e_sym.push_back(qe_sym[e]); e_tgt.push_back(off + tb); }
            }
            st_eend.push_back((int32_t)e_sym.size());
        }
        start_state[q] = off + block[start];
        if (verbose)
            std::fprintf(stderr, "psc_build: q=%d groups=%zu trie=%zu states=%d blocks=%d max-threads=%zu classes=%zu %.1fs\n",
                         q, groups.size(), tn_label.size(), N, nb, max_threads, masks.size(),
                         std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count());
        clear_q();
    }
};

// The union of the per-thread automata (Sec. 3.5: the union over all q is
// what gets minimised).  Mask classes are re-interned globally and state ids
// offset per builder.
struct Automaton {
    std::vector<int32_t> st_cls, st_def, st_ebeg, st_eend, e_sym, e_tgt, start_state;
    Interner<uint32_t> masks;
    int64_t states_built = 0;
};

Automaton merge(std::vector<std::unique_ptr<Builder>> &bs, int32_t nQ, int32_t W) {
    Automaton A;
    A.start_state.assign(nQ, -1);
    std::vector<uint32_t> zero(W, 0);
    bool added;
    A.masks.find_or_add(zero.data(), W, &added);
    for (auto &bp : bs) {
        Builder &B = *bp;
        std::vector<int32_t> cmap(B.masks.size());
        for (size_t c = 0; c < B.masks.size(); c++)
            cmap[c] = A.masks.find_or_add(B.masks.data((int32_t)c), W, &added);
        B.masks.clear();
        int32_t off = (int32_t)A.st_cls.size();
        int32_t eoff = (int32_t)A.e_sym.size();
        for (size_t s = 0; s < B.st_cls.size(); s++) {
            A.st_cls.push_back(cmap[B.st_cls[s]]);
            A.st_def.push_back(off + B.st_def[s]);
            A.st_ebeg.push_back(eoff + B.st_ebeg[s]);
            A.st_eend.push_back(eoff + B.st_eend[s]);
        }
        for (size_t e = 0; e < B.e_sym.size(); e++) {
            A.e_sym.push_back(B.e_sym[e]);
            A.e_tgt.push_back(off + B.e_tgt[e]);
        }
        for (int32_t q = 0; q < nQ; q++)
            if (B.start_state[q] >= 0) A.start_state[q] = off + B.start_state[q];
        A.states_built += B.states_built;
        B.st_cls.clear(); B.st_def.clear(); B.st_ebeg.clear(); B.st_eend.clear();
        B.e_sym.clear(); B.e_tgt.clear();
        B.st_cls.shrink_to_fit(); B.e_sym.shrink_to_fit(); B.e_tgt.shrink_to_fit();
    }
    return A;
}

// ---------------------------------------------------------- minimisation

std::vector<int32_t> minimise(const Automaton &B, int32_t *n_blocks_out) {
    return moore((int32_t)B.st_cls.size(), B.st_cls, B.st_def, B.st_ebeg, B.st_eend, B.e_sym, B.e_tgt,
                 n_blocks_out);
}

}  // namespace

psc_status check_instance(const psc_grammar *g, const psc_vocab *v, std::string *msg) {
    try {
        validate(g, v);
        return PSC_OK;
    } catch (const BuildError &e) {
        *msg = e.what();
        return e.code;
    }
}
}  // namespace psc

using namespace psc;

size_t psc_handle::device_bytes_needed(uint32_t flags) const { return psc::device_layout(*this, flags).total; }

namespace psc {
DeviceLayout device_layout(const psc_handle &h, uint32_t flags) {
    auto up = [](size_t n) { return (n + 255) & ~(size_t)255; };
    DeviceLayout L{};
    L.sliced = (flags & PSC_BIND_SLICED) != 0;
    L.table = table_off(h.n_lex);
    L.masks = L.table + up(h.table.size() * sizeof(int32_t));
    if (L.sliced) {
        L.ids = L.masks + up(h.slices.size() * sizeof(uint32_t));
        L.gram = L.ids + up(h.slice_ids.size() * sizeof(int32_t));
    } else {
        L.ids = L.masks;
        L.gram = L.masks + up(h.masks.size() * sizeof(uint32_t));
    }
    L.vbytes = L.gram + up(h.gram.size() * sizeof(int32_t));
    L.argmax = L.vbytes + up(h.vbytes.size());
    L.packed = L.argmax + kArgmaxBytes;
    L.closure = L.packed + up((size_t)h.n_lr * h.adv.n_term * sizeof(int32_t));
    L.pred = L.closure + up(goto_closure_bytes(h));
    L.total = L.pred + up((size_t)start_block_count(h.n_lex) * kPredInts * sizeof(int32_t));
    return L;
}

void slice_masks(psc_handle &h) {
    const int64_t nc = h.n_classes;
    const int32_t ns = h.mask_stride / kSliceWords;
    h.n_slices = ns;
    h.slice_ids.assign((size_t)nc * ns, 0);
    h.slices.clear();
    // open addressing over the distinct slices, keyed by a 64-bit hash
    size_t cap = 1024;   // a power of two, at least twice the number of slices
    while (cap < (size_t)(nc * ns) * 2) cap <<= 1;
    std::vector<int32_t> slot(cap, -1);
    std::vector<uint64_t> key(cap, 0);
    int32_t n = 0;
    for (int64_t c = 0; c < nc; c++)
        for (int32_t k = 0; k < ns; k++) {
            const uint32_t *w = h.masks.data() + (size_t)c * h.mask_stride + (size_t)k * kSliceWords;
            uint64_t x = 0x9E3779B97F4A7C15ull;
            for (int i = 0; i < kSliceWords; i++) x = mix64(x ^ w[i]);
            size_t at = (size_t)x & (cap - 1);
            int32_t id = -1;
            for (;; at = (at + 1) & (cap - 1)) {
                if (slot[at] < 0) break;
                if (key[at] == x &&
                    std::equal(w, w + kSliceWords, h.slices.data() + (size_t)slot[at] * kSliceWords)) {
                    id = slot[at];
                    break;
                }
            }
            if (id < 0) {
                id = n++;
                slot[at] = id;
                key[at] = x;
                h.slices.insert(h.slices.end(), w, w + kSliceWords);
            }
            h.slice_ids[(size_t)c * ns + k] = id;
        }
    h.n_unique_slices = n;
    h.info.mask_slices_unique = n;
    h.info.sliced_mask_bytes = (int64_t)(h.slices.size() + h.slice_ids.size()) * 4;
}

bool packed_action(const psc_handle &h, std::vector<int32_t> &out) {
    out.clear();
    const AdvanceLayout &L = h.adv;
    const int32_t *act = h.gram.data() + L.action, *lhs = h.gram.data() + L.prod_lhs,
                  *len = h.gram.data() + L.prod_len;
    const int64_t n = (int64_t)h.n_lr * L.n_term;
    std::vector<int32_t> v(act, act + n);
    for (int32_t &a : v) {
        if ((a & 3) != 2) continue;
        const int32_t p = a >> 2;
        if (len[p] > 255 || lhs[p] >= (1 << 21)) return false;
        a = 2 | (len[p] << 2) | (lhs[p] << 10);
    }
    out.swap(v);
    return true;
}

size_t goto_closure_bytes(const psc_handle &h) {
    const size_t n = (size_t)h.n_lr * h.adv.n_nt * h.adv.n_term * sizeof(int32_t);
    return n <= kClosureMaxBytes ? n : 0;
}

void goto_closure(const psc_handle &h, std::vector<int32_t> &out) {
    out.clear();
    if (!goto_closure_bytes(h)) return;
    const AdvanceLayout &L = h.adv;
    const int32_t *act = h.gram.data() + L.action, *go = h.gram.data() + L.go,
                  *lhs = h.gram.data() + L.prod_lhs, *len = h.gram.data() + L.prod_len;
    const int64_t nt = L.n_nt, nT = L.n_term;
    out.assign((size_t)h.n_lr * nt * nT, -1);
    for (int64_t s = 0; s < h.n_lr; s++)
        for (int64_t A = 0; A < nt; A++) {
            const int32_t g0 = go[s * nt + A];
            int32_t *row = out.data() + (s * nt + A) * nT;
            if (g0 < 0) continue;
            for (int64_t t = 0; t < nT; t++) {
                int32_t x = g0;
                int64_t steps = 0;
                for (;;) {
                    const int32_t a = act[(int64_t)x * nT + t];
                    if ((a & 3) != 2 || len[a >> 2] != 1) break;
                    if (++steps > nt) { x = g0; break; }      // a cycle of unit productions: not skipped
                    x = go[s * nt + lhs[a >> 2]];
                    if (x < 0) break;
                }
                row[t] = x;
            }
        }
}

void start_blocks(const psc_handle &h, std::vector<int32_t> &out) {
    const int32_t nb = start_block_count(h.n_lex);
    out.assign((size_t)nb * kStartBlockInts, 0);
    const int64_t T = (int64_t)h.table.size();
    auto at = [&](int64_t i) { return i < T ? h.table[(size_t)i] : 0; };
    for (int32_t q = 0; q < nb; q++) {
        const int32_t ref = h.table[(size_t)q];
        if (ref < 0 || (ref & 3) == kRefDense) continue;
        const int64_t row = ref & ~3;
        int32_t *blk = out.data() + (size_t)q * kStartBlockInts;
        // chain entries and sparse rows are both 16 bytes per lane
        for (int lane = 0; lane < 64; lane++)
            for (int k = 0; k < 4; k++) blk[4 * lane + k] = at(row + 4 * lane + k);
    }
}
}  // namespace psc

namespace {
// Keep the problem instance for the device advance (the lexing and parsing
// steps of Algorithm 2 run on the GPU between classifications).
void copy_advance_tables(psc_handle *h, const psc_grammar *g, const psc_vocab *v) {
    AdvanceLayout &L = h->adv;
    std::vector<int32_t> &B = h->gram;
    auto put = [&](int64_t &at, const int32_t *src, int64_t n) {
        at = (int64_t)B.size();
        B.insert(B.end(), src, src + n);
    };
    put(L.lex_next, g->lex_next, (int64_t)g->n_lex_states * 256);
    put(L.lex_accept, g->lex_accept, g->n_lex_states);
    L.ignored = (int64_t)B.size();
    for (int32_t t = 0; t < g->n_terminals; t++) B.push_back(g->terminal_ignored[t] ? 1 : 0);
    put(L.action, g->action, (int64_t)g->n_lr_states * g->n_terminals);
    put(L.go, g->goto_table, (int64_t)g->n_lr_states * g->n_nonterminals);
    put(L.prod_lhs, g->prod_lhs, g->n_productions);
    put(L.prod_len, g->prod_len, g->n_productions);
    const int64_t total = v->offsets[v->n_tokens];
    if (total >= INT32_MAX) throw BuildError(PSC_E_LIMIT, "vocabulary spellings exceed 2 GiB");
    L.tok_off = (int64_t)B.size();
    for (int32_t t = 0; t <= v->n_tokens; t++) B.push_back((int32_t)v->offsets[t]);
    L.n_term = g->n_terminals;
    L.n_nt = g->n_nonterminals;
    L.end_term = g->end_terminal;
    L.eos = v->eos_id;
    h->vbytes.assign(v->bytes ? v->bytes : nullptr, v->bytes ? v->bytes + total : nullptr);
    if (h->vbytes.empty()) h->vbytes.push_back(0);
}
}  // namespace

extern "C" psc_status psc_build(const psc_grammar *grammar, const psc_vocab *vocab, psc_handle **out) {
    auto t0 = std::chrono::steady_clock::now();
    if (!grammar || !vocab || !out) {
        set_error("psc_build: null argument");
        return PSC_E_INVALID_ARG;
    }
    *out = nullptr;
    try {
        validate(grammar, vocab);
        Gram G{grammar->n_lex_states, grammar->n_terminals, grammar->n_lr_states, grammar->n_nonterminals,
               grammar->n_productions, grammar->end_terminal, grammar->lex_next, grammar->lex_accept,
               grammar->action, grammar->goto_table, grammar->prod_lhs, grammar->prod_len,
               grammar->terminal_ignored};
        bool verbose = std::getenv("PSC_BUILD_VERBOSE") != nullptr;
        Completions C = completions(G);
        VocabTrie VT = vocab_trie(vocab);
        // the CPUs this process may run on (its affinity mask), capped by
        // OMP_NUM_THREADS when that is set; PSC_BUILD_THREADS overrides both
        int32_t n_threads = (int32_t)std::thread::hardware_concurrency();
        cpu_set_t cpus;
        if (sched_getaffinity(0, sizeof(cpus), &cpus) == 0) n_threads = CPU_COUNT(&cpus);
        if (const char *e = std::getenv("OMP_NUM_THREADS")) {
            const int k = std::atoi(e);
            if (k > 0) n_threads = std::min(n_threads, k);
        }
        if (const char *e = std::getenv("PSC_BUILD_THREADS")) n_threads = std::atoi(e);
        n_threads = std::max(1, std::min({n_threads, 32, G.nQ}));
        std::vector<std::unique_ptr<Builder>> builders;
        for (int32_t t = 0; t < n_threads; t++) {
            builders.emplace_back(new Builder(G, vocab, C, VT, verbose));
            builders.back()->start_state.assign(G.nQ, -1);
        }
        std::atomic<int32_t> next_q{0};
        std::atomic<int64_t> total_states{0};
        std::vector<std::exception_ptr> errs(n_threads);
        auto work = [&](int32_t t) {
            try {
                Builder &Bt = *builders[t];
                Bt.total_states = &total_states;
                if (const char *e = std::getenv("PSC_BUILD_MAX_STATES")) Bt.max_states = std::atoll(e);
                for (int32_t q; (q = next_q.fetch_add(1)) < G.nQ;) Bt.build_for_lexer_state(q);
            } catch (...) {
                errs[t] = std::current_exception();
                next_q.store(G.nQ);
            }
        };
        std::vector<std::thread> pool;
        try {
            for (int32_t t = 1; t < n_threads; t++) pool.emplace_back(work, t);
        } catch (const std::system_error &) {
            // fewer threads than asked for: the lexer states are taken from a
            // shared counter, so the threads that did start build all of them
        }
        work(0);
        for (auto &th : pool) th.join();
        for (auto &e : errs)
            if (e) std::rethrow_exception(e);
        Automaton B = merge(builders, G.nQ, (vocab->n_tokens + 31) / 32);
        builders.clear();

        int32_t nb = 0;
        std::vector<int32_t> block = minimise(B, &nb);
        int32_t N = (int32_t)B.st_cls.size();
        std::vector<int32_t> rep(nb, -1);
        for (int32_t s = 0; s < N; s++)
            if (rep[block[s]] < 0) rep[block[s]] = s;

        // minimised automaton: per block, end class, default block, edges
        std::vector<int32_t> m_cls(nb), m_def(nb), m_ebeg(nb + 1);
        std::vector<int32_t> m_sym, m_tgt;
        for (int32_t b = 0; b < nb; b++) {
            int32_t s = rep[b];
            m_cls[b] = B.st_cls[s];
            m_def[b] = block[B.st_def[s]];
            m_ebeg[b] = (int32_t)m_sym.size();
            for (int32_t e = B.st_ebeg[s]; e < B.st_eend[s]; e++) {
                int32_t tb = block[B.e_tgt[e]];
                if (tb != m_def[b]) { m_sym.push_back(B.e_sym[e]); m_tgt.push_back(tb); }
            }
        }
        m_ebeg[nb] = (int32_t)m_sym.size();

        // determined(b): every state reachable from b has the same class.
        // Tarjan's SCCs come out successors-first, so one pass suffices.
        const int32_t MANY = -2, UNSET = -3;
        std::vector<int32_t> det(nb, UNSET), idx(nb, -1), low(nb, 0), comp_stack;
        std::vector<uint8_t> on(nb, 0), in_comp(nb, 0);
        int32_t counter = 0;
        auto succ_count = [&](int32_t b) { return 1 + (m_ebeg[b + 1] - m_ebeg[b]); };
        auto succ_at = [&](int32_t b, int32_t i) { return i == 0 ? m_def[b] : m_tgt[m_ebeg[b] + i - 1]; };
        for (int32_t root = 0; root < nb; root++) {
            if (idx[root] >= 0) continue;
            std::vector<std::pair<int32_t, int32_t>> work{{root, 0}};
            while (!work.empty()) {
                auto &[v, it] = work.back();
                if (it == 0 && idx[v] < 0) {
                    idx[v] = low[v] = counter++;
                    comp_stack.push_back(v);
                    on[v] = 1;
                }
                bool descended = false;
                while (it < succ_count(v)) {
                    int32_t w = succ_at(v, it);
                    it++;
                    if (idx[w] < 0) {
                        work.emplace_back(w, 0);
                        descended = true;
                        break;
                    }
                    if (on[w]) low[v] = std::min(low[v], idx[w]);
                }
                if (descended) continue;
                int32_t vv = v;
                if (low[vv] == idx[vv]) {
                    std::vector<int32_t> members;
                    while (true) {
                        int32_t x = comp_stack.back();
                        comp_stack.pop_back();
                        on[x] = 0;
                        members.push_back(x);
                        if (x == vv) break;
                    }
                    int32_t d = m_cls[members[0]];
                    for (int32_t x : members) in_comp[x] = 1;
                    for (int32_t x : members) {
                        if (m_cls[x] != d) d = MANY;
                        for (int32_t i = 0; i < succ_count(x) && d != MANY; i++) {
                            int32_t w = succ_at(x, i);
                            if (!in_comp[w] && det[w] != d) d = MANY;
                        }
                    }
                    for (int32_t x : members) { det[x] = d; in_comp[x] = 0; }
                }
                work.pop_back();
                if (!work.empty()) {
                    int32_t parent = work.back().first;
                    low[parent] = std::min(low[parent], low[vv]);
                }
            }
        }

        // Canonical order: breadth-first from the start states of q = 0, 1, ...
        // (default successor first, then edges by symbol).  Block and class
        // ids above depend on thread scheduling; everything emitted below is
        // numbered in this order, so the output is identical on every build.
        // Blocks no start state reaches are never walked and are dropped.
        std::vector<int32_t> order;
        {
            std::vector<uint8_t> seen(nb, 0);
            auto push = [&](int32_t b) { if (!seen[b]) { seen[b] = 1; order.push_back(b); } };
            for (int32_t q = 0; q < G.nQ; q++) push(block[B.start_state[q]]);
            for (size_t k = 0; k < order.size(); k++) {
                int32_t b = order[k];
                if (det[b] >= 0) continue;
                push(m_def[b]);
                for (int32_t e = m_ebeg[b]; e < m_ebeg[b + 1]; e++) push(m_tgt[e]);
            }
        }

        // keep only the classes a walk can end in, renumbered densely in the
        // canonical order (class 0, the all-zero row, always keeps id 0)
        std::vector<int32_t> cls_map(B.masks.size(), -1);
        std::vector<int32_t> kept{0};
        cls_map[0] = 0;
        auto keep = [&](int32_t c) {
            if (cls_map[c] < 0) { cls_map[c] = (int32_t)kept.size(); kept.push_back(c); }
            return cls_map[c];
        };
        for (int32_t b : order) {
            m_cls[b] = keep(m_cls[b]);
            if (det[b] >= 0) det[b] = keep(det[b]);
        }

        // flatten
        std::unique_ptr<psc_handle> owned(new psc_handle());
        psc_handle *h = owned.get();
        h->V = vocab->n_tokens;
        h->W = (vocab->n_tokens + 31) / 32;
        h->mask_stride = (h->W + 63) & ~63;   // 256-byte rows
        h->n_lex = G.nQ;
        h->n_lr = G.nPi;
        h->n_classes = (int32_t)kept.size();
        copy_advance_tables(h, grammar, vocab);
        std::vector<int32_t> ref(nb, 0);
        // Thin states (at most two explicit edges) become chain entries.  A
        // thin state moves on along its lowest explicit edge into a thin
        // state, else along its lowest explicit edge, and an edge-free state
        // along its default; chains follow these moves in canonical order.
        const bool use_chains = G.nPi <= kMaxChainAlphabet;
        auto is_thin = [&](int32_t b) { return use_chains && det[b] < 0 && m_ebeg[b + 1] - m_ebeg[b] <= 2; };
        auto cont_edge = [&](int32_t b) -> int32_t {     // edge index, or -1: any symbol (default)
            if (m_ebeg[b + 1] == m_ebeg[b]) return -1;
            for (int32_t e = m_ebeg[b]; e < m_ebeg[b + 1]; e++)
                if (is_thin(m_tgt[e])) return e;
            return m_ebeg[b];
        };
        auto cont_target = [&](int32_t b) { int32_t e = cont_edge(b); return e < 0 ? m_def[b] : m_tgt[e]; };
        std::vector<std::vector<int32_t>> chains;
        {
            std::vector<uint8_t> placed(nb, 0);
            for (int32_t b : order) {
                if (!is_thin(b) || placed[b]) continue;
                std::vector<int32_t> ch{b};
                placed[b] = 1;
                for (int32_t t = cont_target(b); (int)ch.size() < kChainMax && is_thin(t) && !placed[t];
                     t = cont_target(t)) {
                    ch.push_back(t);
                    placed[t] = 1;
                }
                chains.push_back(std::move(ch));
            }
        }
        // A chain shorter than kChainReach goes on with copies of the thin
        // states that follow its last one, so that a walk crossing into the
        // next chain does not pay a load for the jump between them; copies
        // are entries like the originals, but no ref points at them.
        std::vector<std::vector<int32_t>> laid(chains.size());
        std::vector<int32_t> jump_to(chains.size());
        for (size_t c = 0; c < chains.size(); c++) {
            laid[c] = chains[c];
            int32_t t = cont_target(chains[c].back());
            while ((int)laid[c].size() < kChainReach && is_thin(t)) {
                laid[c].push_back(t);
                t = cont_target(t);
            }
            jump_to[c] = t;
        }
        int64_t off = (G.nQ + 3) & ~3;
        h->rows_off = off;
        int32_t rows = 0, dense = 0, max_sparse = 0, chain_states = 0;
        for (int32_t b : order) {
            if (det[b] >= 0) { ref[b] = class_ref(det[b]); continue; }
            rows++;
            if (is_thin(b)) continue;
            int32_t ne = m_ebeg[b + 1] - m_ebeg[b];
            bool is_dense = ne > kSparseMax;
            ref[b] = (int32_t)off | (is_dense ? kRefDense : 0);
            int64_t len = is_dense ? kRowHeader + 2LL * G.nPi : kSparseHeader + (int64_t)kSparseEdge * ne;
            off += (len + 3) & ~3;
            if (is_dense) dense++; else max_sparse = std::max(max_sparse, ne);
            if (off > (1LL << 30)) throw BuildError(PSC_E_LIMIT, "classifier table exceeds 4 GiB");
        }
        h->chains_off = off;
        for (size_t c = 0; c < chains.size(); c++) {
            const auto &ch = chains[c];
            for (size_t j = 0; j < ch.size(); j++) ref[ch[j]] = (int32_t)(off + kChainEntry * j) | kRefChain;
            off += kChainEntry * (int64_t)(laid[c].size() + 1);
            chain_states += (int32_t)ch.size();
            if (off > (1LL << 30)) throw BuildError(PSC_E_LIMIT, "classifier table exceeds 4 GiB");
        }
        h->table_end = off;
        h->table.assign((size_t)off + kTablePad, 0);
        for (int32_t q = 0; q < G.nQ; q++) h->table[q] = ref[block[B.start_state[q]]];
        for (int32_t b : order) {
            if (det[b] >= 0 || is_thin(b)) continue;
            int32_t *row = h->table.data() + ref_offset(ref[b]);
            int32_t ne = m_ebeg[b + 1] - m_ebeg[b];
            row[0] = m_cls[b];
            if (ref_is_dense(ref[b])) {
                row[1] = -1;
                row[2] = ref[m_def[b]];
                row[3] = 0;
                for (int32_t X = 0; X < G.nPi; X++) {
                    row[kRowHeader + 2 * X] = ref[m_def[b]];
                    row[kRowHeader + 2 * X + 1] = kNoSkip;   // set below
                }
                for (int32_t e = m_ebeg[b]; e < m_ebeg[b + 1]; e++) row[kRowHeader + 2 * m_sym[e]] = ref[m_tgt[e]];
            } else {
                row[1] = ne;
                row[2] = row[3] = 0;
                row[4] = kSymNone;
                row[5] = ref[m_def[b]];
                row[6] = kNoSkip;   // set below, once the chains are laid out
                row[7] = 0;
                for (int32_t e = 0; e < ne; e++) {
                    int32_t *en = row + kSparseHeader + kSparseEdge * e;
                    en[0] = m_sym[m_ebeg[b] + e];
                    en[1] = ref[m_tgt[m_ebeg[b] + e]];
                    en[2] = kNoSkip;
                    en[3] = 0;
                }
            }
        }
        for (size_t c = 0; c < chains.size(); c++) {
            int32_t *e = h->table.data() + ref_offset(ref[chains[c][0]]);
            for (int32_t b : laid[c]) {
                const int32_t ce = cont_edge(b);
                uint32_t a = ce < 0 ? (uint32_t)kSymWild : (uint32_t)m_sym[ce], bs = kSymNone;
                int32_t rb = 0;
                for (int32_t k = m_ebeg[b]; k < m_ebeg[b + 1]; k++)
                    if (k != ce) { bs = (uint32_t)m_sym[k]; rb = ref[m_tgt[k]]; }
                e[0] = (int32_t)(a | (bs << 16));
                e[1] = rb;
                e[2] = ref[m_def[b]];
                e[3] = m_cls[b];
                e += kChainEntry;
            }
            e[0] = (int32_t)((uint32_t)kSymJump | ((uint32_t)kSymNone << 16));
            e[1] = 0;
            e[2] = ref[jump_to[c]];
            e[3] = 0;
        }
        // the skips of the rows' refs (sparse defaults and edges, dense entries)
        {
            const int32_t *t = h->table.data();
            const int64_t n = (int64_t)h->table.size();
            int64_t skips = 0;
            for (int32_t b : order) {
                if (det[b] >= 0 || is_thin(b)) continue;
                int32_t *row = h->table.data() + ref_offset(ref[b]);
                if (ref_is_dense(ref[b])) {
                    for (int32_t X = 0; X < G.nPi; X++) {
                        row[kRowHeader + 2 * X + 1] = chain_skip(t, n, row[kRowHeader + 2 * X]);
                        skips += row[kRowHeader + 2 * X + 1] != kNoSkip;
                    }
                    continue;
                }
                row[6] = chain_skip(t, n, row[5]);
                skips += row[6] != kNoSkip;
                for (int32_t e = 0; e < row[1]; e++) {
                    int32_t *en = row + kSparseHeader + kSparseEdge * e;
                    en[2] = chain_skip(t, n, en[1]);
                    skips += en[2] != kNoSkip;
                }
            }
            h->info.skip_edges = skips;
        }
        h->masks.assign((size_t)h->n_classes * h->mask_stride, 0);
        for (int32_t c = 0; c < h->n_classes; c++)
            std::copy(B.masks.data(kept[c]), B.masks.data(kept[c]) + h->W,
                      h->masks.begin() + (size_t)c * h->mask_stride);

        psc_info_t &I = h->info;
        I.vocab_size = h->V;
        I.mask_words = h->W;
        I.mask_stride_words = h->mask_stride;
        I.n_lex_states = G.nQ;
        I.n_lr_states = G.nPi;
        I.n_classes = h->n_classes;
        I.dfa_states_built = B.states_built;
        I.dfa_states = (int32_t)order.size();
        I.dfa_rows = rows;
        I.dense_rows = dense;
        I.max_sparse_edges = max_sparse;
        I.chain_states = chain_states;
        I.chains = (int32_t)chains.size();
        I.table_bytes = (int64_t)h->table.size() * 4;
        I.mask_table_bytes = (int64_t)h->masks.size() * 4;
        slice_masks(*h);
        I.device_bytes = (int64_t)h->device_bytes_needed();
        I.build_seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        *out = owned.release();
        return PSC_OK;
    } catch (const BuildError &e) {
        set_error(std::string("psc_build: ") + e.what());
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("psc_build: out of host memory");
        return PSC_E_OOM;
    } catch (const std::exception &e) {
        // nothing may unwind through the C ABI; what is left is running out
        // of host resources (a table too long for a vector, no thread)
        set_error(std::string("psc_build: out of host resources (") + e.what() + ")");
        return PSC_E_OOM;
    }
}

extern "C" psc_status psc_info(const psc_handle *h, psc_info_t *out) {
    if (!h || !out) {
        set_error("psc_info: null argument");
        return PSC_E_INVALID_ARG;
    }
    *out = h->info;
    return PSC_OK;
}

extern "C" size_t psc_device_bytes(const psc_handle *h) { return h ? h->device_bytes_needed() : 0; }

extern "C" size_t psc_device_bytes_ex(const psc_handle *h, uint32_t flags) {
    return h ? h->device_bytes_needed(flags) : 0;
}

extern "C" psc_status psc_classify_host(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                        const int32_t *lexer_states, int32_t B, int32_t *out_classes) {
    if (!h || B < 0 || (B > 0 && (!stacks || !stack_lens || !lexer_states || !out_classes))) {
        set_error("psc_classify_host: invalid argument");
        return PSC_E_INVALID_ARG;
    }
    const int32_t *T = h->table.data();
    int64_t base = 0;
    for (int32_t b = 0; b < B; b++) {
        int32_t len = stack_lens[b], q = lexer_states[b];
        const int32_t *st = stacks + base;
        base += len > 0 ? len : 0;
        if (len <= 0 || q < 0 || q >= h->n_lex) { out_classes[b] = -1; continue; }
        int32_t ref = T[q];
        int32_t i = len - 1;
        int32_t cls = -1;
        for (;;) {
            if (ref_is_class(ref)) { cls = ref_class(ref); break; }
            const int32_t *row = T + ref_offset(ref);
            if (ref_is_chain(ref)) {                         // one chain entry at a time
                const uint32_t x = (uint32_t)row[0];
                const int32_t a = (int32_t)(x & 0xFFFF), bs = (int32_t)(x >> 16);
                if (a == kSymJump) { ref = row[2]; continue; }
                if (i < 0) { cls = row[3]; break; }
                const int32_t X = st[i--];
                if (X < 0 || X >= h->n_lr) break;
                if (a == kSymWild || X == a) ref = (ref_offset(ref) + kChainEntry) | kRefChain;
                else ref = X == bs ? row[1] : row[2];
                continue;
            }
            if (i < 0) { cls = row[0]; break; }
            const int32_t X = st[i--];
            if (X < 0 || X >= h->n_lr) break;
            int32_t nxt, skip;
            if (ref_is_dense(ref)) {
                nxt = row[kRowHeader + 2 * X];
                skip = row[kRowHeader + 2 * X + 1];
            } else {
                int32_t lo = 0, hi = row[1];
                nxt = row[5];
                skip = row[6];
                while (lo < hi) {
                    const int32_t mid = (lo + hi) / 2;
                    const int32_t *en = row + kSparseHeader + kSparseEdge * mid;
                    if (en[0] == X) { nxt = en[1]; skip = en[2]; break; }
                    if (en[0] < X) lo = mid + 1; else hi = mid;
                }
            }
            ref = nxt;
            // a skip reads its k symbols (in range) without visiting the
            // wildcard entries, as the device walk does
            if (skip != kNoSkip) {
                const int32_t k = (int32_t)((uint32_t)skip >> 27);
                bool ok = i - (k - 1) >= 0;
                for (int32_t j = 0; ok && j < k; j++) ok = st[i - j] >= 0 && st[i - j] < h->n_lr;
                if (ok) {
                    i -= k;
                    ref = (int32_t)(((uint32_t)skip & ((1u << 27) - 1)) - (1u << 26));
                }
            }
        }
        out_classes[b] = cls;
    }
    return PSC_OK;
}

extern "C" psc_status psc_class_mask_host(const psc_handle *h, int32_t cls, uint32_t *out_row) {
    if (!h || !out_row || cls < 0 || cls >= h->n_classes) {
        set_error("psc_class_mask_host: invalid argument");
        return PSC_E_INVALID_ARG;
    }
    std::copy(h->masks.begin() + (size_t)cls * h->mask_stride,
              h->masks.begin() + (size_t)cls * h->mask_stride + h->W, out_row);
    return PSC_OK;
}

extern "C" psc_status psc_host_state(const psc_handle *h, const uint8_t *text, size_t len, int32_t *q,
                                     int32_t *stack, int32_t cap, int32_t *stack_len) {
    if (!h || (len > 0 && !text) || !q || !stack || !stack_len || cap < 1) {
        set_error("psc_host_state: null argument or cap < 1");
        return PSC_E_INVALID_ARG;
    }
    const AdvanceLayout &L = h->adv;
    const int32_t *g = h->gram.data();
    const int32_t *lex_next = g + L.lex_next, *lex_accept = g + L.lex_accept, *ignored = g + L.ignored;
    const int32_t *action = g + L.action, *go = g + L.go, *prod_lhs = g + L.prod_lhs, *prod_len = g + L.prod_len;
    int32_t n = 0;
    auto push = [&](int32_t s) {
        if (n >= cap) return false;
        stack[n++] = s;
        return true;
    };
    // more reductions than this for one terminal means the tables loop
    const int64_t max_steps = (int64_t)(L.n_nt + 2) * (2 * (int64_t)cap + 8) + 65536;
    // one terminal: the reductions its lookahead selects, then its shift
    auto feed = [&](int32_t t) -> psc_status {
        for (int64_t k = 0; k < max_steps; k++) {
            const int32_t a = action[(int64_t)stack[n - 1] * L.n_term + t];
            switch (a & 3) {
            case 1:
                return push(a >> 2) ? PSC_OK : PSC_E_LIMIT;
            case 2: {
                const int32_t p = a >> 2;
                if (prod_len[p] >= n) return PSC_E_NOT_VIABLE;
                n -= prod_len[p];
                const int32_t s = go[(int64_t)stack[n - 1] * L.n_nt + prod_lhs[p]];
                if (s < 0) return PSC_E_NOT_VIABLE;
                if (!push(s)) return PSC_E_LIMIT;
                break;
            }
            default:   // an error entry (accept is only ever reached with $end, never fed here)
                return PSC_E_NOT_VIABLE;
            }
        }
        return PSC_E_GRAMMAR;
    };
    push(0);                     // s0, the parser's start state
    int32_t cur = 0;             // q0: nothing pending
    psc_status st = PSC_OK;
    for (size_t i = 0; i < len && st == PSC_OK; i++) {
        const uint8_t c = text[i];
        const int32_t nx = lex_next[(int64_t)cur * 256 + c];
        if (nx >= 0) {
            cur = nx;
            continue;
        }
        // the pending lexeme ends here: it must be a terminal, and c starts the next one
        const int32_t t = cur != 0 ? lex_accept[cur] : -1;
        if (t < 0) {
            st = PSC_E_NOT_VIABLE;
            break;
        }
        if (!ignored[t]) st = feed(t);
        cur = lex_next[c];
        if (st == PSC_OK && cur < 0) st = PSC_E_NOT_VIABLE;
    }
    if (st != PSC_OK) {
        set_error(st == PSC_E_NOT_VIABLE ? "psc_host_state: the text is not a viable prefix"
                  : st == PSC_E_LIMIT    ? "psc_host_state: the stack would exceed cap"
                                         : "psc_host_state: the parser tables loop");
        return st;
    }
    *q = cur;
    *stack_len = n;
    return PSC_OK;
}

extern "C" void psc_free(psc_handle *h) { delete h; }

extern "C" const char *psc_last_error(void) { return g_last_error.c_str(); }
