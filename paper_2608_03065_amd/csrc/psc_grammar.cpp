// psc_grammar.cpp -- grammar text -> the problem instance of Algorithm 1.
//
// Algorithm 1 takes the lexer T (a finite-state transducer over bytes,
// Sec. 2.2) and the parser P (a deterministic pushdown automaton, realised
// as LR tables, Sec. 2.4 and Sec. 4.1) as given.  Sec. 4.1 obtains them from
// an LALR(1) generator before the method starts; this file is that step,
// behind the C ABI: psc_grammar_compile turns grammar text into the tables
// psc_build takes, and reports any LALR(1) conflict instead of resolving it
// (the method covers deterministic grammars only, Sec. 5.3).
//
// Lexer: each terminal is a regular expression or a literal; the union is
// compiled to one byte DFA (Thompson NFA, subset construction over byte
// equivalence classes, removal of states that reach no accepting state,
// Moore minimisation with q0 kept alone as state 0).  Lexing is longest
// match with one byte of lookahead; two terminals matching the same longest
// lexeme are resolved by explicit priority, then literal over regex, then
// declaration order.
//
// Parser: the LR(0) automaton (kernels numbered breadth-first, moves taken in
// symbol order: nonterminals by id, then terminals by id) with LALR(1)
// lookaheads by DeRemer and Pennello's relations (reads, includes,
// lookback).  Reductions are never defaulted.
//
// The grammar text (one statement per line; '#' starts a comment outside
// quotes and slashes):
//   %start NAME                 the start nonterminal
//   %ignore NAME /regex/        a terminal the lexer consumes and drops
//   %literal "text" [PRIO]      declare a literal terminal at this point
//   NAME[.PRIO]: /regex/        a regex terminal
//   name: item item ...         a production; items are declared terminal
//   name: a | b c |             names, "literals" (declared on first use) or
//       | d                     nonterminals; '|' separates alternatives, an
//                               empty alternative is the empty production; a
//                               line starting with '|' continues the rule.
// Literals take the escapes \\ \" \n \t \r \xHH.  Regexes are over bytes:
// . [...] [^...] ( ) (?: ) | * + ? {m} {m,} {m,n} and the escapes \n \t \r
// \f \v \0 \xHH \d \w \s; any other escaped byte stands for itself, so \/
// is a slash.  Terminal ids follow declaration order, then $END; nonterminal
// ids follow the order of first appearance as a rule's left side, then the
// augmented start $start; production 0 is $start -> start.

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <memory>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "psc_internal.hpp"

using psc::set_error;

namespace {

struct CompileError {
    psc_status code;
    std::string msg;
};

[[noreturn]] void fail(psc_status code, const std::string &msg) { throw CompileError{code, msg}; }

// Bounds that keep hostile text from exhausting the stack or memory.
constexpr int kMaxRegexDepth = 500;        // nested groups in one regex
constexpr size_t kMaxNfaStates = 4000000;  // all terminals together
constexpr size_t kMaxDfaStates = 1000000;  // before minimisation
constexpr size_t kMaxSubsetTotal = 200000000;   // NFA states summed over the DFA's subsets

// ---------------------------------------------------------------- byte sets

struct ByteSet {
    uint64_t w[4] = {0, 0, 0, 0};
    void add(int b) { w[b >> 6] |= 1ull << (b & 63); }
    bool has(int b) const { return (w[b >> 6] >> (b & 63)) & 1; }
    void add_range(int lo, int hi) {
        for (int b = lo; b <= hi; b++) add(b);
    }
    ByteSet &operator|=(const ByteSet &o) {
        for (int k = 0; k < 4; k++) w[k] |= o.w[k];
        return *this;
    }
    ByteSet complement() const {
        ByteSet r;
        for (int k = 0; k < 4; k++) r.w[k] = ~w[k];
        return r;
    }
    int count() const { return __builtin_popcountll(w[0]) + __builtin_popcountll(w[1]) +
                               __builtin_popcountll(w[2]) + __builtin_popcountll(w[3]); }
    int highest() const {
        for (int k = 3; k >= 0; k--)
            if (w[k]) return k * 64 + 63 - __builtin_clzll(w[k]);
        return -1;
    }
    static ByteSet one(int b) {
        ByteSet s;
        s.add(b);
        return s;
    }
};

ByteSet digit_set() {
    ByteSet s;
    s.add_range('0', '9');
    return s;
}
ByteSet word_set() {
    ByteSet s = digit_set();
    s.add_range('A', 'Z');
    s.add_range('a', 'z');
    s.add('_');
    return s;
}
ByteSet space_set() {
    ByteSet s;
    for (int b : {0x20, 0x09, 0x0A, 0x0D, 0x0B, 0x0C}) s.add(b);
    return s;
}

// ---------------------------------------------------------------- regex AST

struct Node {
    enum Kind { Set, Cat, Alt, Star, Plus, Opt, Rep } kind;
    ByteSet set;
    std::vector<int> kids;
    int lo = 0, hi = -1;   // Rep: hi < 0 means unbounded
};

class RegexParser {
  public:
    RegexParser(const std::string &p, std::vector<Node> &nodes) : p_(p), nodes_(nodes) {}

    int parse() {
        const int n = alt();
        if (i_ != p_.size()) bad("unexpected '" + std::string(1, p_[i_]) + "' at " + std::to_string(i_));
        return n;
    }

  private:
    const std::string &p_;
    std::vector<Node> &nodes_;
    size_t i_ = 0;
    int depth_ = 0;

    [[noreturn]] void bad(const std::string &m) const { fail(PSC_E_GRAMMAR, "regex /" + p_ + "/: " + m); }
    int peek() const { return i_ < p_.size() ? (unsigned char)p_[i_] : -1; }
    int take() {
        if (i_ >= p_.size()) bad("unexpected end");
        return (unsigned char)p_[i_++];
    }
    int add(Node n) {
        nodes_.push_back(std::move(n));
        return (int)nodes_.size() - 1;
    }
    int set_node(const ByteSet &s) {
        Node n{Node::Set};
        n.set = s;
        return add(std::move(n));
    }

    int alt() {
        std::vector<int> parts{cat()};
        while (peek() == '|') {
            take();
            parts.push_back(cat());
        }
        if (parts.size() == 1) return parts[0];
        Node n{Node::Alt};
        n.kids = std::move(parts);
        return add(std::move(n));
    }

    int cat() {
        std::vector<int> parts;
        while (peek() >= 0 && peek() != '|' && peek() != ')') parts.push_back(repeat());
        if (parts.size() == 1) return parts[0];
        Node n{Node::Cat};
        n.kids = std::move(parts);
        return add(std::move(n));
    }

    static int parse_int(const std::string &s, bool &ok) {
        size_t a = 0, b = s.size();
        while (a < b && s[a] == ' ') a++;
        while (b > a && s[b - 1] == ' ') b--;
        ok = a < b;
        long v = 0;
        for (size_t k = a; k < b && ok; k++) {
            if (s[k] < '0' || s[k] > '9') ok = false;
            else v = v * 10 + (s[k] - '0');
            if (v > 100000) ok = false;
        }
        return (int)v;
    }

    int repeat() {
        int node = atom();
        for (int ops = 0;; ops++) {
            if (ops > kMaxRegexDepth) bad("more than " + std::to_string(kMaxRegexDepth) + " repetition operators in a row");
            const int c = peek();
            if (c == '*' || c == '+' || c == '?') {
                take();
                Node n{c == '*' ? Node::Star : c == '+' ? Node::Plus : Node::Opt};
                n.kids = {node};
                node = add(std::move(n));
            } else if (c == '{') {
                const size_t j = p_.find('}', i_);
                if (j == std::string::npos) bad("missing }");
                const std::string body = p_.substr(i_ + 1, j - i_ - 1);
                i_ = j + 1;
                Node n{Node::Rep};
                n.kids = {node};
                bool ok = true, ok2 = true;
                const size_t comma = body.find(',');
                if (comma != std::string::npos) {
                    n.lo = parse_int(body.substr(0, comma), ok);
                    const std::string rest = body.substr(comma + 1);
                    if (rest.find_first_not_of(' ') == std::string::npos) n.hi = -1;
                    else n.hi = parse_int(rest, ok2);
                } else {
                    n.lo = n.hi = parse_int(body, ok);
                }
                if (!ok || !ok2 || (n.hi >= 0 && n.hi < n.lo)) bad("bad repetition {" + body + "}");
                node = add(std::move(n));
            } else {
                return node;
            }
        }
    }

    static int hexval(int c) {
        if (c >= '0' && c <= '9') return c - '0';
        if (c >= 'a' && c <= 'f') return c - 'a' + 10;
        if (c >= 'A' && c <= 'F') return c - 'A' + 10;
        return -1;
    }

    ByteSet escape() {
        const int c = take();
        switch (c) {
        case 'n': return ByteSet::one(0x0A);
        case 't': return ByteSet::one(0x09);
        case 'r': return ByteSet::one(0x0D);
        case 'f': return ByteSet::one(0x0C);
        case 'v': return ByteSet::one(0x0B);
        case '0': return ByteSet::one(0x00);
        case 'd': return digit_set();
        case 'w': return word_set();
        case 's': return space_set();
        case 'x': {
            const int h1 = i_ < p_.size() ? hexval((unsigned char)p_[i_]) : -1;
            const int h2 = i_ + 1 < p_.size() ? hexval((unsigned char)p_[i_ + 1]) : -1;
            if (h1 < 0 || h2 < 0) bad("bad \\x escape");
            i_ += 2;
            return ByteSet::one(h1 * 16 + h2);
        }
        default: return ByteSet::one(c);
        }
    }

    int atom() {
        const int c = take();
        if (c == '(') {
            if (p_.compare(i_, 2, "?:") == 0) i_ += 2;
            if (++depth_ > kMaxRegexDepth) bad("groups nested deeper than " + std::to_string(kMaxRegexDepth));
            const int n = alt();
            depth_--;
            if (peek() != ')') bad("missing )");
            take();
            return n;
        }
        if (c == '[') return set_node(char_class());
        if (c == '.') return set_node(ByteSet::one(0x0A).complement());
        if (c == '\\') return set_node(escape());
        if (c == '*' || c == '+' || c == '?' || c == '{') bad("nothing to repeat at " + std::to_string(i_ - 1));
        return set_node(ByteSet::one(c));
    }

    ByteSet char_class() {
        bool neg = false;
        if (peek() == '^') {
            take();
            neg = true;
        }
        ByteSet m;
        bool first = true;
        for (;;) {
            const int c = peek();
            if (c < 0) bad("unterminated class");
            if (c == ']' && !first) {
                take();
                break;
            }
            first = false;
            ByteSet lo_m;
            take();
            lo_m = c == '\\' ? escape() : ByteSet::one(c);
            if (peek() == '-' && i_ + 1 < p_.size() && p_[i_ + 1] != ']') {
                take();
                const int hc = take();
                const ByteSet hi_m = hc == '\\' ? escape() : ByteSet::one(hc);
                const int lo = lo_m.highest(), hi = hi_m.highest();
                if (lo_m.count() != 1 || hi_m.count() != 1 || hi < lo) bad("bad range");
                m.add_range(lo, hi);
            } else {
                m |= lo_m;
            }
        }
        return neg ? m.complement() : m;
    }
};

// ---------------------------------------------------------------- lexer DFA

struct Terminal {
    std::string name;
    int ast = -1;
    int priority = 0;
    bool literal = false;
    bool ignored = false;
};

struct Nfa {
    std::vector<std::vector<int>> eps;
    std::vector<std::vector<std::pair<ByteSet, int>>> edges;
    std::vector<int> accept;   // terminal id per state, -1

    int make() {
        if (eps.size() >= kMaxNfaStates)
            fail(PSC_E_LIMIT, "the terminals' NFA exceeds " + std::to_string(kMaxNfaStates) + " states");
        eps.emplace_back();
        edges.emplace_back();
        accept.push_back(-1);
        return (int)eps.size() - 1;
    }

    // a fresh fragment (start, end) for AST node n
    std::pair<int, int> frag(const std::vector<Node> &nodes, int n) {
        const Node &nd = nodes[n];
        switch (nd.kind) {
        case Node::Set: {
            const int s = make(), e = make();
            edges[s].push_back({nd.set, e});
            return {s, e};
        }
        case Node::Cat: {
            const int s = make();
            int cur = s;
            for (int k : nd.kids) {
                const auto ab = frag(nodes, k);
                eps[cur].push_back(ab.first);
                cur = ab.second;
            }
            return {s, cur};
        }
        case Node::Alt: {
            const int s = make(), e = make();
            for (int k : nd.kids) {
                const auto ab = frag(nodes, k);
                eps[s].push_back(ab.first);
                eps[ab.second].push_back(e);
            }
            return {s, e};
        }
        case Node::Star:
        case Node::Plus:
        case Node::Opt: {
            const int s = make(), e = make();
            const auto ab = frag(nodes, nd.kids[0]);
            eps[s].push_back(ab.first);
            eps[ab.second].push_back(e);
            if (nd.kind != Node::Plus) eps[s].push_back(e);
            if (nd.kind != Node::Opt) eps[ab.second].push_back(ab.first);
            return {s, e};
        }
        case Node::Rep: {
            // lo copies, then either a star or (hi - lo) optional copies
            const int s = make();
            int cur = s;
            auto chain = [&](std::pair<int, int> ab) {
                eps[cur].push_back(ab.first);
                cur = ab.second;
            };
            for (int k = 0; k < nd.lo; k++) chain(frag(nodes, nd.kids[0]));
            auto wrapped = [&](bool star) {
                const int ws = make(), we = make();
                const auto ab = frag(nodes, nd.kids[0]);
                eps[ws].push_back(ab.first);
                eps[ab.second].push_back(we);
                eps[ws].push_back(we);
                if (star) eps[ab.second].push_back(ab.first);
                return std::make_pair(ws, we);
            };
            if (nd.hi < 0) chain(wrapped(true));
            else
                for (int k = nd.lo; k < nd.hi; k++) chain(wrapped(false));
            return {s, cur};
        }
        }
        fail(PSC_E_GRAMMAR, "internal: bad regex node");
    }
};

struct VecHash {
    size_t operator()(const std::vector<int> &v) const {
        uint64_t h = 1469598103934665603ull;
        for (int x : v) h = (h ^ (uint32_t)x) * 1099511628211ull;
        return (size_t)h;
    }
};

struct Lexer {
    int n_states = 0;
    std::vector<int32_t> next;     // [n_states][256]
    std::vector<int32_t> accept;   // [n_states]
};

Lexer build_lexer(const std::vector<Terminal> &terms, const std::vector<Node> &nodes) {
    Nfa nfa;
    const int master = nfa.make();
    for (size_t t = 0; t < terms.size(); t++) {
        const auto se = nfa.frag(nodes, terms[t].ast);
        nfa.eps[master].push_back(se.first);
        nfa.accept[se.second] = (int)t;
    }
    // the larger rank wins a tie on the same lexeme
    auto better = [&](int a, int b) {   // is terminal a ranked above terminal b?
        if (terms[a].priority != terms[b].priority) return terms[a].priority > terms[b].priority;
        if (terms[a].literal != terms[b].literal) return terms[a].literal;
        return a < b;
    };

    // byte classes: bytes that no edge set tells apart
    std::vector<const ByteSet *> sets;
    for (const auto &row : nfa.edges)
        for (const auto &e : row) sets.push_back(&e.first);
    std::vector<int> cls_of(256);
    std::vector<int> reps;
    {
        std::map<std::vector<uint64_t>, int> sig;
        const size_t nw = (sets.size() + 63) / 64;
        for (int b = 0; b < 256; b++) {
            std::vector<uint64_t> key(nw, 0);
            for (size_t k = 0; k < sets.size(); k++)
                if (sets[k]->has(b)) key[k >> 6] |= 1ull << (k & 63);
            auto it = sig.find(key);
            if (it == sig.end()) {
                it = sig.emplace(std::move(key), (int)reps.size()).first;
                reps.push_back(b);
            }
            cls_of[b] = it->second;
        }
    }
    const int n_cls = (int)reps.size();

    // subset construction; the move of a subset on a byte class is the
    // epsilon closure of its edges' targets, taken as one search over the
    // whole target set (one visited array, told apart by a stamp), so a move
    // costs the size of its result and not the sum of overlapping closures
    const int n_nfa = (int)nfa.eps.size();
    std::vector<uint32_t> seen(n_nfa, 0);
    uint32_t stamp = 0;
    size_t subset_total = 0;
    auto close = [&](std::vector<int> &set) {
        ++stamp;
        std::vector<int> out;
        out.reserve(set.size());
        for (int v : set)
            if (seen[v] != stamp) {
                seen[v] = stamp;
                out.push_back(v);
            }
        for (size_t k = 0; k < out.size(); k++)
            for (int w : nfa.eps[out[k]])
                if (seen[w] != stamp) {
                    seen[w] = stamp;
                    out.push_back(w);
                }
        std::sort(out.begin(), out.end());
        set = std::move(out);
    };

    std::unordered_map<std::vector<int>, int, VecHash> ids;
    std::vector<std::vector<int>> order;
    std::vector<int> trans, acc;
    {
        std::vector<int> s0{master};
        close(s0);
        subset_total = s0.size();
        ids.emplace(s0, 0);
        order.push_back(std::move(s0));
    }
    for (size_t i = 0; i < order.size(); i++) {
        const std::vector<int> cur = order[i];
        int best = -1;
        for (int s : cur) {
            const int t = nfa.accept[s];
            if (t >= 0 && (best < 0 || better(t, best))) best = t;
        }
        acc.push_back(best);
        std::vector<std::pair<const ByteSet *, int>> edges;
        for (int u : cur)
            for (const auto &e : nfa.edges[u]) edges.push_back({&e.first, e.second});
        for (int c = 0; c < n_cls; c++) {
            const int b = reps[c];
            std::vector<int> tgt;
            for (const auto &e : edges)
                if (e.first->has(b)) tgt.push_back(e.second);
            if (tgt.empty()) {
                trans.push_back(-1);
                continue;
            }
            close(tgt);
            auto it = ids.find(tgt);
            int j;
            if (it == ids.end()) {
                j = (int)order.size();
                subset_total += tgt.size();
                if (order.size() + 1 > kMaxDfaStates || subset_total > kMaxSubsetTotal)
                    fail(PSC_E_LIMIT, "the lexer DFA exceeds " + std::to_string(kMaxDfaStates) + " states or " +
                                          std::to_string(kMaxSubsetTotal) + " NFA states over all its subsets");
                ids.emplace(tgt, j);
                order.push_back(std::move(tgt));
            } else {
                j = it->second;
            }
            trans.push_back(j);
        }
    }
    if (acc[0] >= 0) fail(PSC_E_GRAMMAR, "terminal " + terms[acc[0]].name + " matches the empty string");

    // drop states from which no accepting state is reachable (q0 kept): a
    // search backwards from the accepting states over the reversed moves
    int n = (int)order.size();
    std::vector<char> live(n, 0);
    {
        std::vector<int> rstart(n + 1, 0), redge;
        for (size_t k = 0; k < trans.size(); k++)
            if (trans[k] >= 0) rstart[trans[k] + 1]++;
        for (int s = 0; s < n; s++) rstart[s + 1] += rstart[s];
        redge.resize(rstart[n]);
        std::vector<int> fill(rstart.begin(), rstart.end() - 1);
        for (int s = 0; s < n; s++)
            for (int c = 0; c < n_cls; c++) {
                const int t = trans[(size_t)s * n_cls + c];
                if (t >= 0) redge[fill[t]++] = s;
            }
        std::vector<int> work;
        for (int s = 0; s < n; s++)
            if (acc[s] >= 0) {
                live[s] = 1;
                work.push_back(s);
            }
        while (!work.empty()) {
            const int t = work.back();
            work.pop_back();
            for (int k = rstart[t]; k < rstart[t + 1]; k++)
                if (!live[redge[k]]) {
                    live[redge[k]] = 1;
                    work.push_back(redge[k]);
                }
        }
    }
    live[0] = 1;
    std::vector<int> remap(n, -1), keep;
    for (int s = 0; s < n; s++)
        if (live[s]) {
            remap[s] = (int)keep.size();
            keep.push_back(s);
        }
    std::vector<int> T((size_t)keep.size() * n_cls), A(keep.size());
    for (size_t k = 0; k < keep.size(); k++) {
        A[k] = acc[keep[k]];
        for (int c = 0; c < n_cls; c++) {
            const int t = trans[(size_t)keep[k] * n_cls + c];
            T[k * n_cls + c] = t >= 0 ? remap[t] : -1;
        }
    }
    n = (int)keep.size();

    // Moore refinement: q0 alone, the others by accepted terminal
    std::vector<int> block(n);
    {
        std::map<int, int> first;
        for (int s = 0; s < n; s++) {
            const int key = s == 0 ? -2 : A[s];
            block[s] = first.emplace(key, (int)first.size()).first->second;
        }
    }
    int n_blocks = 0;
    for (int b : block) n_blocks = std::max(n_blocks, b + 1);
    for (;;) {
        std::map<std::vector<int>, int> sig;
        std::vector<int> nb(n);
        for (int s = 0; s < n; s++) {
            std::vector<int> key(n_cls + 1);
            key[0] = block[s];
            for (int c = 0; c < n_cls; c++) {
                const int t = T[(size_t)s * n_cls + c];
                key[c + 1] = t >= 0 ? block[t] : -1;
            }
            nb[s] = sig.emplace(std::move(key), (int)sig.size()).first->second;
        }
        const int cnt = (int)sig.size();
        block = std::move(nb);
        if (cnt == n_blocks) break;
        n_blocks = cnt;
    }
    // renumber blocks by first occurrence (q0's block is 0)
    std::vector<int> num(n_blocks, -1), rep(n_blocks, -1);
    int next_id = 0;
    for (int s = 0; s < n; s++)
        if (num[block[s]] < 0) {
            num[block[s]] = next_id++;
            rep[num[block[s]]] = s;
        }
    Lexer L;
    L.n_states = n_blocks;
    L.next.assign((size_t)n_blocks * 256, -1);
    L.accept.assign(n_blocks, -1);
    for (int q = 0; q < n_blocks; q++) {
        const int s = rep[q];
        L.accept[q] = A[s];
        for (int b = 0; b < 256; b++) {
            const int t = T[(size_t)s * n_cls + cls_of[b]];
            L.next[(size_t)q * 256 + b] = t >= 0 ? num[block[t]] : -1;
        }
    }
    return L;
}

// ---------------------------------------------------------------- LALR(1)

// A symbol as a sortable key: nonterminals (by id) before terminals (by id).
constexpr int kTermBit = 1 << 30;
inline bool is_term(int sym) { return (sym & kTermBit) != 0; }
inline int sym_id(int sym) { return sym & ~kTermBit; }

struct Production {
    int lhs;
    std::vector<int> body;   // symbol keys
};

struct Bits {
    std::vector<uint64_t> w;
    explicit Bits(int n = 0) : w((size_t)(n + 63) / 64, 0) {}
    void set(int i) { w[i >> 6] |= 1ull << (i & 63); }
    bool test(int i) const { return (w[i >> 6] >> (i & 63)) & 1; }
    void operator|=(const Bits &o) {
        for (size_t k = 0; k < w.size(); k++) w[k] |= o.w[k];
    }
};

// DeRemer and Pennello's digraph: F(x) = init(x) | U{F(y) : x rel y}, with
// every member of a strongly connected component given the component's union.
std::vector<Bits> digraph(const std::vector<std::vector<int>> &rel, std::vector<Bits> F) {
    const int n = (int)F.size();
    const int kDone = 1 << 30;
    std::vector<int> N(n, 0), depth(n, 0), stack;
    for (int root = 0; root < n; root++) {
        if (N[root]) continue;
        std::vector<std::pair<int, size_t>> work{{root, 0}};
        while (!work.empty()) {
            auto [x, it] = work.back();
            work.pop_back();
            if (it == 0) {
                stack.push_back(x);
                depth[x] = (int)stack.size();
                N[x] = depth[x];
            } else {
                const int y = rel[x][it - 1];
                N[x] = std::min(N[x], N[y]);
                F[x] |= F[y];
            }
            bool descended = false;
            while (it < rel[x].size()) {
                const int y = rel[x][it++];
                if (N[y] == 0) {
                    work.push_back({x, it});
                    work.push_back({y, 0});
                    descended = true;
                    break;
                }
                N[x] = std::min(N[x], N[y]);
                F[x] |= F[y];
            }
            if (descended) continue;
            if (N[x] == depth[x]) {
                for (;;) {
                    const int top = stack.back();
                    stack.pop_back();
                    N[top] = kDone;
                    if (top != x) F[top] = F[x];
                    if (top == x) break;
                }
            }
        }
    }
    return F;
}

struct Tables {
    int n_states = 0;
    std::vector<int32_t> action, go;
};

Tables lalr1(const std::vector<Production> &prods, int n_terms, int n_nts, int end_id,
             const std::vector<std::string> &term_names, const std::vector<std::string> &nt_names) {
    std::vector<std::vector<int>> by_lhs(n_nts);
    for (size_t p = 0; p < prods.size(); p++) by_lhs[prods[p].lhs].push_back((int)p);

    std::vector<char> nullable(n_nts, 0);
    for (bool changed = true; changed;) {
        changed = false;
        for (const auto &pr : prods) {
            if (nullable[pr.lhs]) continue;
            bool all = true;
            for (int s : pr.body)
                if (is_term(s) || !nullable[sym_id(s)]) {
                    all = false;
                    break;
                }
            if (all) {
                nullable[pr.lhs] = 1;
                changed = true;
            }
        }
    }

    // nonterminals whose productions enter the closure of an item before nt
    std::vector<std::vector<int>> nt_closure(n_nts);
    for (int nt = 0; nt < n_nts; nt++) {
        std::vector<char> seen(n_nts, 0);
        std::vector<int> out{nt};
        seen[nt] = 1;
        for (size_t k = 0; k < out.size(); k++)
            for (int p : by_lhs[out[k]]) {
                const auto &b = prods[p].body;
                if (!b.empty() && !is_term(b[0]) && !seen[sym_id(b[0])]) {
                    seen[sym_id(b[0])] = 1;
                    out.push_back(sym_id(b[0]));
                }
            }
        nt_closure[nt] = std::move(out);
    }
    typedef std::pair<int, int> Item;   // (production, dot)
    auto closure = [&](const std::vector<Item> &kernel) {
        std::vector<Item> items = kernel;
        std::vector<char> need(n_nts, 0);
        for (const auto &it : kernel) {
            const auto &b = prods[it.first].body;
            if (it.second < (int)b.size() && !is_term(b[it.second]))
                for (int a : nt_closure[sym_id(b[it.second])]) need[a] = 1;
        }
        for (int a = 0; a < n_nts; a++)
            if (need[a])
                for (int p : by_lhs[a]) items.push_back({p, 0});
        return items;
    };

    std::map<std::vector<Item>, int> state_of;
    std::vector<std::vector<Item>> kernels{{{0, 0}}};
    state_of.emplace(kernels[0], 0);
    std::vector<std::map<int, int>> trans;
    for (size_t i = 0; i < kernels.size(); i++) {
        std::map<int, std::vector<Item>> moves;
        for (const auto &it : closure(kernels[i])) {
            const auto &b = prods[it.first].body;
            if (it.second < (int)b.size()) moves[b[it.second]].push_back({it.first, it.second + 1});
        }
        std::map<int, int> row;
        for (auto &mv : moves) {
            std::vector<Item> k = mv.second;
            std::sort(k.begin(), k.end());
            k.erase(std::unique(k.begin(), k.end()), k.end());
            auto f = state_of.find(k);
            int j;
            if (f == state_of.end()) {
                j = (int)kernels.size();
                state_of.emplace(k, j);
                kernels.push_back(std::move(k));
            } else {
                j = f->second;
            }
            row[mv.first] = j;
        }
        trans.push_back(std::move(row));
    }
    const int n_states = (int)kernels.size();

    // nonterminal transitions and the DeRemer-Pennello relations
    std::vector<std::pair<int, int>> nt_trans;
    std::map<std::pair<int, int>, int> nt_trans_id;
    for (int s = 0; s < n_states; s++)
        for (const auto &kv : trans[s])
            if (!is_term(kv.first)) {
                nt_trans_id[{s, sym_id(kv.first)}] = (int)nt_trans.size();
                nt_trans.push_back({s, sym_id(kv.first)});
            }
    const int start_nt = sym_id(prods[0].body[0]);
    std::vector<Bits> DR(nt_trans.size(), Bits(n_terms));
    std::vector<std::vector<int>> reads(nt_trans.size());
    for (size_t idx = 0; idx < nt_trans.size(); idx++) {
        const auto [p, A] = nt_trans[idx];
        const int r = trans[p].at(A);
        for (const auto &kv : trans[r]) {
            if (is_term(kv.first)) DR[idx].set(sym_id(kv.first));
            else if (nullable[sym_id(kv.first)]) reads[idx].push_back(nt_trans_id.at({r, sym_id(kv.first)}));
        }
        if (p == 0 && A == start_nt) DR[idx].set(end_id);
    }
    const std::vector<Bits> Read = digraph(reads, DR);

    std::vector<std::vector<int>> includes(nt_trans.size());
    std::map<std::pair<int, int>, std::vector<int>> lookback;
    for (size_t idx = 0; idx < nt_trans.size(); idx++) {
        const auto [pp, B] = nt_trans[idx];
        for (int prod : by_lhs[B]) {
            const auto &body = prods[prod].body;
            int s = pp;
            for (size_t pos = 0; pos < body.size(); pos++) {
                const int sym = body[pos];
                if (!is_term(sym)) {
                    bool rest_nullable = true;
                    for (size_t r = pos + 1; r < body.size(); r++)
                        if (is_term(body[r]) || !nullable[sym_id(body[r])]) {
                            rest_nullable = false;
                            break;
                        }
                    if (rest_nullable) includes[nt_trans_id.at({s, sym_id(sym)})].push_back((int)idx);
                }
                s = trans[s].at(sym);
            }
            lookback[{s, prod}].push_back((int)idx);
        }
    }
    const std::vector<Bits> Follow = digraph(includes, Read);

    Tables Tb;
    Tb.n_states = n_states;
    Tb.action.assign((size_t)n_states * n_terms, 0);
    Tb.go.assign((size_t)n_states * n_nts, -1);
    struct Conflict {
        int state, term, had, want;
    };
    std::vector<Conflict> conflicts;
    for (int s = 0; s < n_states; s++) {
        for (const auto &kv : trans[s]) {
            if (is_term(kv.first)) Tb.action[(size_t)s * n_terms + sym_id(kv.first)] = (kv.second << 2) | 1;
            else Tb.go[(size_t)s * n_nts + sym_id(kv.first)] = kv.second;
        }
        for (const auto &it : closure(kernels[s])) {
            if (it.second != (int)prods[it.first].body.size()) continue;
            Bits la(n_terms);
            int want;
            if (it.first == 0) {
                want = 3;
                la.set(end_id);
            } else {
                want = (it.first << 2) | 2;
                auto f = lookback.find({s, it.first});
                if (f != lookback.end())
                    for (int idx : f->second) la |= Follow[idx];
            }
            for (int t = 0; t < n_terms; t++) {
                if (!la.test(t)) continue;
                int32_t &a = Tb.action[(size_t)s * n_terms + t];
                if (a != 0 && a != want) conflicts.push_back({s, t, a, want});
                else a = want;
            }
        }
    }
    if (!conflicts.empty()) {
        auto show = [&](int a) {
            const int k = a & 3;
            if (k == 1) return "shift " + std::to_string(a >> 2);
            if (k == 3) return std::string("accept");
            std::string r = "reduce " + nt_names[prods[a >> 2].lhs] + " ->";
            for (int sym : prods[a >> 2].body)
                r += " " + (is_term(sym) ? term_names[sym_id(sym)] : nt_names[sym_id(sym)]);
            return r;
        };
        std::string msg = std::to_string(conflicts.size()) + " LALR(1) conflicts; first:";
        for (size_t k = 0; k < conflicts.size() && k < 5; k++)
            msg += " [state " + std::to_string(conflicts[k].state) + " on " + term_names[conflicts[k].term] +
                   ": " + show(conflicts[k].had) + " | " + show(conflicts[k].want) + "]";
        fail(PSC_E_NOT_LALR1, msg);
    }
    return Tb;
}

// ---------------------------------------------------------------- grammar text

class TextParser {
  public:
    std::vector<Node> nodes;
    std::vector<Terminal> terms;
    std::unordered_map<std::string, int> term_index;
    std::string start;
    struct Rule {
        std::string lhs;
        std::vector<std::string> body;   // terminal names ('"..."' for literals) or nonterminal names
        int line;
    };
    std::vector<Rule> rules;

    void parse(const char *text, size_t len) {
        size_t pos = 0;
        int line = 0;
        std::string cur_lhs;
        while (pos < len) {
            size_t e = pos;
            while (e < len && text[e] != '\n') e++;
            line++;
            std::string ln(text + pos, e - pos);
            pos = e + 1;
            line_ = line;
            s_ = &ln;
            i_ = 0;
            skip();
            if (at_end()) continue;
            const char c = (*s_)[i_];
            if (c == '%') {
                directive();
                cur_lhs.clear();
            } else if (c == '|') {
                if (cur_lhs.empty()) bad("'|' without a rule to continue");
                i_++;
                alternatives(cur_lhs);
            } else {
                std::string name = ident();
                int prio = 0;
                bool has_prio = false;
                if (peek() == '.') {
                    i_++;
                    prio = integer();
                    has_prio = true;
                }
                skip();
                if (peek() != ':') bad("expected ':' after " + name);
                i_++;
                skip();
                if (peek() == '/') {
                    declare(Terminal{name, parse_regex(slashed()), prio, false, false});
                    end_of_line();
                    cur_lhs.clear();
                } else {
                    if (has_prio) bad("a priority is for terminals only");
                    cur_lhs = name;
                    alternatives(name);
                }
            }
        }
        if (start.empty()) fail(PSC_E_GRAMMAR, "grammar text: no %start");
    }

  private:
    const std::string *s_ = nullptr;
    size_t i_ = 0;
    int line_ = 0;

    [[noreturn]] void bad(const std::string &m) const {
        fail(PSC_E_GRAMMAR, "grammar text, line " + std::to_string(line_) + ": " + m);
    }
    bool at_end() const { return i_ >= s_->size() || (*s_)[i_] == '#'; }
    int peek() const { return i_ < s_->size() ? (unsigned char)(*s_)[i_] : -1; }
    void skip() {
        while (i_ < s_->size() && ((*s_)[i_] == ' ' || (*s_)[i_] == '\t' || (*s_)[i_] == '\r')) i_++;
    }
    void end_of_line() {
        skip();
        if (!at_end()) bad("unexpected text after the statement");
    }
    static bool ident_char(int c) {
        return (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z') || (c >= '0' && c <= '9') || c == '_' || c == '$';
    }
    std::string ident() {
        const size_t a = i_;
        while (i_ < s_->size() && ident_char((unsigned char)(*s_)[i_])) i_++;
        if (a == i_) bad("expected a name");
        return s_->substr(a, i_ - a);
    }
    int integer() {
        bool neg = false;
        if (peek() == '-') {
            neg = true;
            i_++;
        }
        const size_t a = i_;
        long v = 0;
        while (i_ < s_->size() && (*s_)[i_] >= '0' && (*s_)[i_] <= '9' && v < 1000000) v = v * 10 + ((*s_)[i_++] - '0');
        if (a == i_ || v >= 1000000) bad("expected an integer");
        return (int)(neg ? -v : v);
    }
    static int hexval(int c) {
        if (c >= '0' && c <= '9') return c - '0';
        if (c >= 'a' && c <= 'f') return c - 'a' + 10;
        if (c >= 'A' && c <= 'F') return c - 'A' + 10;
        return -1;
    }
    // "..." with escapes -> the literal's bytes
    std::string quoted() {
        i_++;   // opening quote
        std::string out;
        for (;;) {
            if (i_ >= s_->size()) bad("unterminated literal");
            char c = (*s_)[i_++];
            if (c == '"') break;
            if (c == '\\') {
                if (i_ >= s_->size()) bad("unterminated literal");
                const char d = (*s_)[i_++];
                if (d == 'n') c = '\n';
                else if (d == 't') c = '\t';
                else if (d == 'r') c = '\r';
                else if (d == '\\' || d == '"') c = d;
                else if (d == 'x') {
                    const int h1 = i_ < s_->size() ? hexval((unsigned char)(*s_)[i_]) : -1;
                    const int h2 = i_ + 1 < s_->size() ? hexval((unsigned char)(*s_)[i_ + 1]) : -1;
                    if (h1 < 0 || h2 < 0) bad("bad \\x escape in a literal");
                    i_ += 2;
                    c = (char)(h1 * 16 + h2);
                } else {
                    bad(std::string("unknown escape \\") + d + " in a literal");
                }
            }
            out.push_back(c);
        }
        if (out.empty()) bad("empty literal");
        return out;
    }
    // /.../ -> the pattern text, escapes kept (the regex parser reads them)
    std::string slashed() {
        i_++;
        const size_t a = i_;
        while (i_ < s_->size() && (*s_)[i_] != '/') i_ += (*s_)[i_] == '\\' ? 2 : 1;
        if (i_ >= s_->size()) bad("unterminated regex");
        std::string p = s_->substr(a, i_ - a);
        i_++;
        return p;
    }
    int parse_regex(const std::string &pattern) {
        RegexParser rp(pattern, nodes);
        return rp.parse();
    }
    void declare(Terminal t) {
        if (term_index.count(t.name)) bad("terminal " + t.name + " declared twice");
        term_index.emplace(t.name, (int)terms.size());
        terms.push_back(std::move(t));
    }
    std::string literal_term(const std::string &text, int prio) {
        const std::string name = "\"" + text + "\"";
        if (!term_index.count(name)) {
            Node cat{Node::Cat};
            for (unsigned char ch : text) {
                Node n{Node::Set};
                n.set = ByteSet::one(ch);
                nodes.push_back(std::move(n));
                cat.kids.push_back((int)nodes.size() - 1);
            }
            nodes.push_back(std::move(cat));
            term_index.emplace(name, (int)terms.size());
            terms.push_back(Terminal{name, (int)nodes.size() - 1, prio, true, false});
        }
        return name;
    }
    void directive() {
        i_++;
        const std::string d = ident();
        skip();
        if (d == "start") {
            if (!start.empty()) bad("%start given twice");
            start = ident();
        } else if (d == "ignore") {
            const std::string name = ident();
            skip();
            if (peek() != '/') bad("%ignore NAME /regex/");
            declare(Terminal{name, parse_regex(slashed()), 0, false, true});
        } else if (d == "literal") {
            if (peek() != '"') bad("%literal \"text\" [priority]");
            const std::string text = quoted();
            skip();
            const int prio = (peek() == '-' || (peek() >= '0' && peek() <= '9')) ? integer() : 0;
            literal_term(text, prio);
        } else {
            bad("unknown directive %" + d);
        }
        end_of_line();
    }
    void alternatives(const std::string &lhs) {
        std::vector<std::string> body;
        for (;;) {
            skip();
            if (at_end()) break;
            const int c = peek();
            if (c == '|') {
                i_++;
                rules.push_back({lhs, body, line_});
                body.clear();
            } else if (c == '"') {
                body.push_back(literal_term(quoted(), 0));
            } else {
                body.push_back(ident());
            }
        }
        rules.push_back({lhs, body, line_});
    }
};

// The compiled problem instance, owned by the handle.
}  // namespace

struct psc_compiled_grammar {
    Lexer lexer;
    std::vector<uint8_t> ignored;
    int32_t end_terminal = 0;
    Tables parser;
    std::vector<int32_t> prod_lhs, prod_len;
    std::vector<std::string> terminal_names, nonterminal_names;
    int32_t n_terminals = 0, n_nonterminals = 0;
};

namespace {

psc_compiled_grammar *compile_text(const char *text, size_t len) {
    TextParser tp;
    tp.parse(text, len);
    if (tp.terms.empty()) fail(PSC_E_GRAMMAR, "grammar text: no terminals");
    auto G = std::make_unique<psc_compiled_grammar>();
    G->lexer = build_lexer(tp.terms, tp.nodes);
    const int n_decl = (int)tp.terms.size();
    for (const auto &t : tp.terms) {
        G->terminal_names.push_back(t.name);
        G->ignored.push_back(t.ignored ? 1 : 0);
    }
    G->terminal_names.push_back("$END");
    G->ignored.push_back(0);
    G->end_terminal = n_decl;
    G->n_terminals = n_decl + 1;

    std::unordered_map<std::string, int> nt_index;
    for (const auto &r : tp.rules)
        if (!nt_index.count(r.lhs)) {
            if (tp.term_index.count(r.lhs)) fail(PSC_E_GRAMMAR, r.lhs + " is a terminal and a rule's left side");
            nt_index.emplace(r.lhs, (int)G->nonterminal_names.size());
            G->nonterminal_names.push_back(r.lhs);
        }
    if (!nt_index.count(tp.start)) fail(PSC_E_GRAMMAR, "start symbol " + tp.start + " has no rules");
    const int aug = (int)G->nonterminal_names.size();
    G->nonterminal_names.push_back("$start");
    G->n_nonterminals = aug + 1;

    std::vector<Production> prods{{aug, {nt_index.at(tp.start)}}};
    for (const auto &r : tp.rules) {
        Production p{nt_index.at(r.lhs), {}};
        for (const auto &s : r.body) {
            auto t = tp.term_index.find(s);
            if (t != tp.term_index.end()) {
                if (tp.terms[t->second].ignored)
                    fail(PSC_E_GRAMMAR, "line " + std::to_string(r.line) + ": ignored terminal " + s + " used in a rule");
                p.body.push_back(t->second | kTermBit);
                continue;
            }
            auto n = nt_index.find(s);
            if (n == nt_index.end()) fail(PSC_E_GRAMMAR, "line " + std::to_string(r.line) + ": undefined symbol " + s);
            p.body.push_back(n->second);
        }
        prods.push_back(std::move(p));
    }
    G->parser = lalr1(prods, G->n_terminals, G->n_nonterminals, G->end_terminal, G->terminal_names,
                      G->nonterminal_names);
    for (const auto &p : prods) {
        G->prod_lhs.push_back(p.lhs);
        G->prod_len.push_back((int32_t)p.body.size());
    }
    return G.release();
}

}  // namespace

extern "C" psc_status psc_grammar_compile(const char *text, size_t len, psc_compiled_grammar **out) {
    if (!out || (!text && len > 0)) {
        set_error("psc_grammar_compile: null argument");
        return PSC_E_INVALID_ARG;
    }
    *out = nullptr;
    try {
        *out = compile_text(text ? text : "", len);
        return PSC_OK;
    } catch (const CompileError &e) {
        set_error("psc_grammar_compile: " + e.msg);
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("psc_grammar_compile: out of host memory");
        return PSC_E_OOM;
    } catch (const std::exception &e) {
        set_error(std::string("psc_grammar_compile: ") + e.what());
        return PSC_E_GRAMMAR;
    }
}

extern "C" psc_status psc_grammar_view(const psc_compiled_grammar *g, psc_grammar *out) {
    if (!g || !out) {
        set_error("psc_grammar_view: null argument");
        return PSC_E_INVALID_ARG;
    }
    out->n_lex_states = g->lexer.n_states;
    out->lex_next = g->lexer.next.data();
    out->lex_accept = g->lexer.accept.data();
    out->n_terminals = g->n_terminals;
    out->terminal_ignored = g->ignored.data();
    out->end_terminal = g->end_terminal;
    out->n_lr_states = g->parser.n_states;
    out->n_nonterminals = g->n_nonterminals;
    out->action = g->parser.action.data();
    out->goto_table = g->parser.go.data();
    out->n_productions = (int32_t)g->prod_lhs.size();
    out->prod_lhs = g->prod_lhs.data();
    out->prod_len = g->prod_len.data();
    return PSC_OK;
}

extern "C" const char *psc_grammar_symbol_name(const psc_compiled_grammar *g, int32_t terminal, int32_t id) {
    if (!g || id < 0) return nullptr;
    const auto &names = terminal ? g->terminal_names : g->nonterminal_names;
    return id < (int32_t)names.size() ? names[id].c_str() : nullptr;
}

extern "C" void psc_grammar_free(psc_compiled_grammar *g) { delete g; }

extern "C" psc_status psc_build_from_text(const char *text, size_t len, const psc_vocab *vocab, psc_handle **out) {
    if (!out || !vocab) {
        set_error("psc_build_from_text: null argument");
        return PSC_E_INVALID_ARG;
    }
    *out = nullptr;
    psc_compiled_grammar *g = nullptr;
    const psc_status st = psc_grammar_compile(text, len, &g);
    if (st != PSC_OK) return st;
    psc_grammar view;
    psc_grammar_view(g, &view);
    const psc_status b = psc_build(&view, vocab, out);
    psc_grammar_free(g);
    return b;
}
