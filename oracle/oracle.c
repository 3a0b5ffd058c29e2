/*
 * Brute-force grammar-constrained-decoding checker.  TEST INFRASTRUCTURE.
 *
 * Only the tests, the smoke entry point and the benchmark's CPU-baseline leg
 * load this file.  It shares no code with the classifier construction or the
 * GPU kernels: it reads the same problem instance (lexer DFA, LR tables,
 * vocabulary, prefix state) and decides every token one at a time, the
 * "naive" method that the paper's Fig. 1b contrasts with the classifier.
 *
 * What is computed.  For a prefix x with lexer state q and parser stack
 * alpha (Sec. 3.2), token v is allowed iff some realizable terminal sequence
 * w in R_q(v) (Sec. 3.1) takes the parser from alpha to a stable stack
 * (eq. simp).  R_q(v) is x' T_p where lexing v from q emits x' and stops in
 * state p, and T_p is the set of terminals the pending lexeme can still
 * become (Sec. 3.1).  The paper proves (Theorems 1-3) that the classifier
 * returns exactly this set, so it is the oracle's definition.
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *  - lexing is longest match with one byte of lookahead, no backtracking;
 *    state 0 is q0 (nothing pending) and is never accepting;
 *  - ignored terminals are consumed by the lexer and never reach the parser;
 *  - T_p is {winner(r) : r accepting and reachable from p}, plus "nothing"
 *    when p = q0 or an ignored terminal is reachable;
 *  - a terminal is processed by running the LR reductions its lookahead
 *    selects and must end in a shift (accept for $end); reductions alone
 *    never make a terminal valid;
 *  - EOS has an empty spelling; it is allowed iff the pending lexeme can end
 *    here (q0, or an accepting state) and the parser then accepts $end,
 *    i.e. iff x itself is in the language;
 *  - a stack view that would pop below the bottom of alpha fails.
 *
 * Masks are packed LSB-first into uint32 words, W = ceil(V/32), tail bits 0.
 *
 * It also advances a prefix state by one token (oracle_advance): the new
 * state after x.v is what lexing v from q and feeding the terminals it emits
 * leaves behind, with the last lexeme still pending in the lexer state
 * (Sec. 3.2: the prefix state is the lexer state plus the parser stack).
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC -o liboracle.so oracle.c
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int32_t n_lex;                 /* |Q|, state 0 = q0                       */
    const int32_t *lex_next;       /* [n_lex][256], -1 = no transition        */
    const int32_t *lex_accept;     /* [n_lex], winning terminal or -1         */
    int32_t n_term;                /* |Gamma| including $end                  */
    const uint8_t *ignored;        /* [n_term]                                */
    int32_t end_term;              /* id of $end                              */
    int32_t n_lr;                  /* |Pi|                                    */
    int32_t n_nt;
    const int32_t *action;         /* [n_lr][n_term], (a&3): 0 err 1 shift 2 reduce 3 accept */
    const int32_t *go;             /* [n_lr][n_nt], -1 = none                 */
    const int32_t *prod_lhs;
    const int32_t *prod_len;
} or_grammar;

typedef struct {
    or_grammar g;
    const uint8_t *vbytes;         /* concatenated token spellings            */
    const int64_t *voffs;          /* [V+1]                                   */
    int32_t V, eos;
    int32_t words_per_set;         /* uint64 words per terminal set           */
    uint64_t *reach;               /* [n_lex][words_per_set]: T_p as a bitset */
    uint8_t *reach_eps;            /* [n_lex]: T_p contains "nothing"         */
} oracle_ctx;

/* ---------------------------------------------------------------------
 * T_p for every lexer state p (Sec. 3.1): the least fixpoint of
 *   reach(p) = {winner(p) if p accepting} U  U_c reach(next(p, c)).
 * Solved by plain iteration until nothing changes.
 * ------------------------------------------------------------------- */
static void compute_completions(oracle_ctx *o) {
    const or_grammar *g = &o->g;
    int32_t n = g->n_lex, W = o->words_per_set;
    o->reach = (uint64_t *)calloc((size_t)n * W, sizeof(uint64_t));
    o->reach_eps = (uint8_t *)calloc((size_t)n, 1);
    for (int32_t p = 0; p < n; p++) {
        int32_t t = g->lex_accept[p];
        if (t >= 0) o->reach[(int64_t)p * W + t / 64] |= 1ull << (t % 64);
    }
    int changed = 1;
    while (changed) {
        changed = 0;
        for (int32_t p = n - 1; p >= 0; p--) {
            uint64_t *rp = o->reach + (int64_t)p * W;
            for (int c = 0; c < 256; c++) {
                int32_t r = g->lex_next[(int64_t)p * 256 + c];
                if (r < 0 || r == p) continue;
                const uint64_t *rr = o->reach + (int64_t)r * W;
                for (int32_t k = 0; k < W; k++) {
                    uint64_t nv = rp[k] | rr[k];
                    if (nv != rp[k]) { rp[k] = nv; changed = 1; }
                }
            }
        }
    }
    for (int32_t p = 0; p < n; p++) {
        if (p == 0) { o->reach_eps[p] = 1; continue; }
        for (int32_t t = 0; t < g->n_term; t++)
            if (g->ignored[t] && (o->reach[(int64_t)p * W + t / 64] >> (t % 64) & 1))
                o->reach_eps[p] = 1;
    }
}

/* ---------------------------------------------------------------------
 * A read-only view of alpha plus a private overlay of pushed states.
 * alpha is stored bottom -> top; `depth` symbols of it are still present.
 * ------------------------------------------------------------------- */
#define OVERLAY_CAP 8192
typedef struct {
    const int32_t *alpha;
    int32_t depth;
    int32_t n;                      /* overlay size */
    int32_t s[OVERLAY_CAP];         /* overlay, bottom -> top */
} view;

static int view_top(const view *v, int32_t *out) {
    if (v->n > 0) { *out = v->s[v->n - 1]; return 1; }
    if (v->depth > 0) { *out = v->alpha[v->depth - 1]; return 1; }
    return 0;
}

static int view_pop(view *v, int32_t m) {
    int32_t from_overlay = m < v->n ? m : v->n;
    v->n -= from_overlay;
    m -= from_overlay;
    if (m > v->depth) return 0;
    v->depth -= m;
    return 1;
}

static void view_push(view *v, int32_t s) {
    if (v->n >= OVERLAY_CAP) {
        fprintf(stderr, "oracle: overlay capacity exceeded\n");
        abort();
    }
    v->s[v->n++] = s;
}

/* Process one terminal t on the parser (the LR reading of a DPDA step,
 * Sec. 2.4): apply the reductions selected by lookahead t, then shift t.
 * Returns 1 iff t was shifted (or $end accepted). */
static int feed(const or_grammar *g, view *v, int32_t t) {
    for (;;) {
        int32_t top;
        if (!view_top(v, &top)) return 0;
        int32_t a = g->action[(int64_t)top * g->n_term + t];
        int kind = a & 3;
        if (kind == 1) { view_push(v, a >> 2); return 1; }
        if (kind == 3) return 1;
        if (kind == 0) return 0;
        int32_t p = a >> 2;
        if (!view_pop(v, g->prod_len[p])) return 0;
        int32_t base;
        if (!view_top(v, &base)) return 0;
        int32_t nx = g->go[(int64_t)base * g->n_nt + g->prod_lhs[p]];
        if (nx < 0) return 0;
        view_push(v, nx);
    }
}

/* Is token `tok` in c(x) for the prefix state (q, alpha)?  eq. simp. */
static int token_allowed(const oracle_ctx *o, int32_t q, const int32_t *alpha, int32_t len,
                         int32_t tok, view *v, view *scratch) {
    const or_grammar *g = &o->g;
    v->alpha = alpha;
    v->depth = len;
    v->n = 0;
    int32_t cur = q;

    if (tok == o->eos) {
        if (cur != 0) {
            int32_t t = g->lex_accept[cur];
            if (t < 0) return 0;
            if (!g->ignored[t] && !feed(g, v, t)) return 0;
        }
        return feed(g, v, g->end_term);
    }

    /* lex the token's bytes from q, feeding every emitted terminal */
    for (int64_t i = o->voffs[tok]; i < o->voffs[tok + 1]; i++) {
        uint8_t c = o->vbytes[i];
        int32_t nx = g->lex_next[(int64_t)cur * 256 + c];
        if (nx >= 0) { cur = nx; continue; }
        if (cur == 0) return 0;
        int32_t t = g->lex_accept[cur];
        if (t < 0) return 0;
        if (!g->ignored[t] && !feed(g, v, t)) return 0;
        cur = g->lex_next[c];
        if (cur < 0) return 0;
    }

    /* the pending lexeme must be able to become a terminal that is shifted */
    if (o->reach_eps[cur]) return 1;
    const uint64_t *rs = o->reach + (int64_t)cur * o->words_per_set;
    for (int32_t t = 0; t < g->n_term; t++) {
        if (!(rs[t / 64] >> (t % 64) & 1)) continue;
        scratch->alpha = v->alpha;
        scratch->depth = v->depth;
        scratch->n = v->n;
        memcpy(scratch->s, v->s, (size_t)v->n * sizeof(int32_t));
        if (feed(g, scratch, t)) return 1;
    }
    return 0;
}

/* ------------------------------------------------------------------ API */

void *oracle_new(const or_grammar *g, const uint8_t *vbytes, const int64_t *voffs, int32_t V,
                 int32_t eos) {
    oracle_ctx *o = (oracle_ctx *)calloc(1, sizeof(oracle_ctx));
    o->g = *g;
    o->vbytes = vbytes;
    o->voffs = voffs;
    o->V = V;
    o->eos = eos;
    o->words_per_set = (g->n_term + 63) / 64;
    compute_completions(o);
    return o;
}

void oracle_free(void *p) {
    oracle_ctx *o = (oracle_ctx *)p;
    if (!o) return;
    free(o->reach);
    free(o->reach_eps);
    free(o);
}

/* Full masks for B prefix states; stacks are ragged (offsets given).
 * Returns the number of OpenMP threads used. */
int oracle_masks(const void *ctx, const int32_t *stacks, const int64_t *offs,
                 const int32_t *lens, const int32_t *qs, int32_t B, uint32_t *out,
                 int32_t n_threads) {
    const oracle_ctx *o = (const oracle_ctx *)ctx;
    int32_t W = (o->V + 31) / 32;
    int used = 1;
    memset(out, 0, (size_t)B * W * sizeof(uint32_t));
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#endif
#pragma omp parallel
    {
#ifdef _OPENMP
#pragma omp single
        used = omp_get_num_threads();
#endif
        view *v = (view *)malloc(sizeof(view));
        view *sc = (view *)malloc(sizeof(view));
#pragma omp for schedule(dynamic, 1) collapse(2)
        for (int32_t b = 0; b < B; b++) {
            for (int32_t w = 0; w < W; w++) {
                uint32_t word = 0;
                for (int32_t j = 0; j < 32; j++) {
                    int32_t tok = w * 32 + j;
                    if (tok >= o->V) break;
                    if (token_allowed(o, qs[b], stacks + offs[b], lens[b], tok, v, sc))
                        word |= 1u << j;
                }
                out[(int64_t)b * W + w] = word;
            }
        }
        free(v);
        free(sc);
    }
    return used;
}

/* Bits for selected tokens of one prefix state (sampled checks). */
void oracle_token_bits(const void *ctx, const int32_t *alpha, int32_t len, int32_t q,
                       const int32_t *toks, int64_t n, uint8_t *out) {
    const oracle_ctx *o = (const oracle_ctx *)ctx;
    view *v = (view *)malloc(sizeof(view));
    view *sc = (view *)malloc(sizeof(view));
    for (int64_t i = 0; i < n; i++) out[i] = (uint8_t)token_allowed(o, q, alpha, len, toks[i], v, sc);
    free(v);
    free(sc);
}

/* The prefix state after one more token (Sec. 3.2; Alg. 2's lexing and
 * parsing steps, which produce the next (q, alpha)).  Lex tok's bytes from q
 * and feed every emitted terminal; the lexeme pending after the last byte
 * stays in the lexer state and is not fed.  EOS feeds the pending lexeme's
 * terminal (if any) and then $end.  Returns
 *   0  advanced: (*q_out, out[0 .. *len_out)) is the new state;
 *   1  rejected: the lexer has no move, or an emitted terminal is not shifted
 *      (this does not look ahead: a token can be advanced over and still leave
 *      a pending lexeme that nothing completes -- the mask rejects those);
 *   2  EOS accepted: x is a sentence of the language (state unchanged);
 *   3  the new stack would be longer than cap. */
int oracle_advance(const void *ctx, int32_t q, const int32_t *alpha, int32_t len, int32_t tok, int32_t cap,
                   int32_t *q_out, int32_t *out, int32_t *len_out) {
    const oracle_ctx *o = (const oracle_ctx *)ctx;
    const or_grammar *g = &o->g;
    view *v = (view *)malloc(sizeof(view));
    v->alpha = alpha;
    v->depth = len;
    v->n = 0;
    int32_t cur = q;
    int status = 0;
    if (tok == o->eos) {
        status = 2;
        if (cur != 0) {
            int32_t t = g->lex_accept[cur];
            if (t < 0 || (!g->ignored[t] && !feed(g, v, t))) status = 1;
        }
        if (status == 2 && !feed(g, v, g->end_term)) status = 1;
        free(v);
        return status;
    }
    for (int64_t i = o->voffs[tok]; i < o->voffs[tok + 1] && status == 0; i++) {
        uint8_t c = o->vbytes[i];
        int32_t nx = g->lex_next[(int64_t)cur * 256 + c];
        if (nx >= 0) { cur = nx; continue; }
        if (cur == 0 || g->lex_accept[cur] < 0) { status = 1; break; }
        int32_t t = g->lex_accept[cur];
        if (!g->ignored[t] && !feed(g, v, t)) { status = 1; break; }
        cur = g->lex_next[c];
        if (cur < 0) status = 1;
    }
    if (status == 0) {
        if (v->depth + v->n > cap) {
            status = 3;
        } else {
            memcpy(out, alpha, (size_t)v->depth * sizeof(int32_t));
            memcpy(out + v->depth, v->s, (size_t)v->n * sizeof(int32_t));
            *len_out = v->depth + v->n;
            *q_out = cur;
        }
    }
    free(v);
    return status;
}
