/*
 * Host lexer + LR parser for producing the hot path's inputs.
 *
 * Given a prefix x, run the lexer from q0 to get the emitted terminals z and
 * the lexer state q, then run the parser from its initial stack on z to get
 * the stack alpha (Sec. 3.2 "Overview of syntactic preprocessing";
 * Algorithm 2, lexing and parsing steps).  The pair (q, alpha) is what the
 * classifier walk consumes.  This file is part of the seeded-input side: it
 * contains no stack-classification arithmetic.
 *
 * Lexing rule: longest match with one byte of lookahead, no backtracking.
 * On a byte with no transition, an accepting state emits its terminal (unless
 * the terminal is ignored) and lexing restarts from q0 on the same byte.
 * Action encoding: (a & 3) 0 error, 1 shift to a>>2, 2 reduce by a>>2,
 * 3 accept.
 *
 * Build: gcc -O2 -shared -fPIC -o _hoststate.so hoststate.c
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    int32_t n_lex;
    const int32_t *lex_next;      /* [n_lex][256] */
    const int32_t *lex_accept;    /* [n_lex] */
    int32_t n_term;
    const uint8_t *ignored;       /* [n_term] */
    int32_t end_term;
    int32_t n_lr;
    int32_t n_nt;
    const int32_t *action;        /* [n_lr][n_term] */
    const int32_t *go;            /* [n_lr][n_nt] */
    const int32_t *prod_lhs;
    const int32_t *prod_len;
} hs_grammar;

enum { HS_OK = 0, HS_LEX_ERROR = 1, HS_SYNTAX_ERROR = 2, HS_CAPACITY = 3, HS_INCOMPLETE = 4 };

typedef struct {
    int32_t *s;
    int64_t n, cap;
} stk;

static int stk_push(stk *st, int32_t v) {
    if (st->n == st->cap) {
        int64_t nc = st->cap ? st->cap * 2 : 256;
        int32_t *ns = (int32_t *)realloc(st->s, (size_t)nc * sizeof(int32_t));
        if (!ns) return 0;
        st->s = ns;
        st->cap = nc;
    }
    st->s[st->n++] = v;
    return 1;
}

/* Feed terminal t to the LR parser: run reductions, then shift or accept.
 * Returns 1 when t was shifted (or accepted for $end), 0 on a syntax error. */
static int feed(const hs_grammar *g, stk *st, int32_t t) {
    for (;;) {
        if (st->n <= 0) return 0;
        int32_t top = st->s[st->n - 1];
        int32_t a = g->action[(int64_t)top * g->n_term + t];
        switch (a & 3) {
        case 1:
            return stk_push(st, a >> 2);
        case 3:
            return 1;
        case 2: {
            int32_t p = a >> 2;
            int32_t m = g->prod_len[p];
            if (st->n - m < 1) return 0;
            st->n -= m;
            int32_t base = st->s[st->n - 1];
            int32_t nx = g->go[(int64_t)base * g->n_nt + g->prod_lhs[p]];
            if (nx < 0) return 0;
            if (!stk_push(st, nx)) return 0;
            break;
        }
        default:
            return 0;
        }
    }
}

/* One byte through the lexer; emits at most one terminal into the parser. */
static int lex_byte(const hs_grammar *g, int32_t *cur, stk *st, uint8_t c) {
    int32_t nx = g->lex_next[(int64_t)(*cur) * 256 + c];
    if (nx >= 0) {
        *cur = nx;
        return HS_OK;
    }
    if (*cur != 0 && g->lex_accept[*cur] >= 0) {
        int32_t t = g->lex_accept[*cur];
        if (!g->ignored[t] && !feed(g, st, t)) return HS_SYNTAX_ERROR;
        nx = g->lex_next[c];
        if (nx < 0) return HS_LEX_ERROR;
        *cur = nx;
        return HS_OK;
    }
    return HS_LEX_ERROR;
}

/* Prefix states at sorted cut positions of one text.
 * For every cut i, the prefix text[0 .. cuts[i]) gives (q_out[i], stack
 * written bottom->top at stacks_out[offs_out[i] ..], lens_out[i]).
 * Stacks are written into a caller buffer of cap_total int32; offs_out[i]
 * is where stack i starts.  Returns HS_OK or the first error (cuts after an
 * error are left with lens_out = 0). */
int hs_prefix_states_at(const hs_grammar *g, const uint8_t *text, int64_t len,
                        const int64_t *cuts, int32_t n_cuts, int32_t *q_out,
                        int32_t *stacks_out, int64_t cap_total, int64_t *offs_out,
                        int32_t *lens_out) {
    stk st = {0, 0, 0};
    int rc = HS_OK;
    int32_t cur = 0;
    int64_t pos = 0, used = 0;
    if (!stk_push(&st, 0)) return HS_CAPACITY;
    for (int32_t i = 0; i < n_cuts; i++) lens_out[i] = 0;
    for (int32_t i = 0; i < n_cuts; i++) {
        int64_t cut = cuts[i];
        if (cut < pos || cut > len) { rc = HS_CAPACITY; break; }
        while (pos < cut) {
            rc = lex_byte(g, &cur, &st, text[pos]);
            if (rc != HS_OK) goto done;
            pos++;
        }
        if (used + st.n > cap_total) { rc = HS_CAPACITY; goto done; }
        memcpy(stacks_out + used, st.s, (size_t)st.n * sizeof(int32_t));
        offs_out[i] = used;
        lens_out[i] = (int32_t)st.n;
        q_out[i] = cur;
        used += st.n;
    }
done:
    free(st.s);
    return rc;
}

/* Single prefix -> (q, stack). */
int hs_prefix_state(const hs_grammar *g, const uint8_t *text, int64_t len, int32_t *q_out,
                    int32_t *stack_out, int32_t cap, int32_t *len_out) {
    int64_t cut = len, off = 0;
    return hs_prefix_states_at(g, text, len, &cut, 1, q_out, stack_out, cap, &off, len_out);
}

/* Whole-string membership: x in L iff lexing ends in q0 or in an accepting
 * state whose terminal is fed, and $end is then accepted. */
int hs_accepts(const hs_grammar *g, const uint8_t *text, int64_t len) {
    stk st = {0, 0, 0};
    int32_t cur = 0;
    int ok = 0;
    if (!stk_push(&st, 0)) return 0;
    for (int64_t i = 0; i < len; i++)
        if (lex_byte(g, &cur, &st, text[i]) != HS_OK) goto done;
    if (cur != 0) {
        int32_t t = g->lex_accept[cur];
        if (t < 0) goto done;
        if (!g->ignored[t] && !feed(g, &st, t)) goto done;
    }
    ok = feed(g, &st, g->end_term);
done:
    free(st.s);
    return ok;
}

/* Batch membership over a ragged list of strings. */
void hs_accepts_batch(const hs_grammar *g, const uint8_t *bytes, const int64_t *offsets,
                      int64_t n, uint8_t *out) {
    for (int64_t i = 0; i < n; i++)
        out[i] = (uint8_t)hs_accepts(g, bytes + offsets[i], offsets[i + 1] - offsets[i]);
}

/* Viable-prefix test: the prefix lexes and parses without error. */
void hs_viable_batch(const hs_grammar *g, const uint8_t *bytes, const int64_t *offsets,
                     int64_t n, uint8_t *out) {
    for (int64_t i = 0; i < n; i++) {
        stk st = {0, 0, 0};
        int32_t cur = 0;
        int ok = stk_push(&st, 0);
        for (int64_t k = offsets[i]; ok && k < offsets[i + 1]; k++)
            ok = lex_byte(g, &cur, &st, bytes[k]) == HS_OK;
        out[i] = (uint8_t)ok;
        free(st.s);
    }
}

/* Stack length after every prefix text[0..i), i = 0..len (depths has len+1
 * entries).  Returns HS_OK or the first error (later depths are -1). */
int hs_depths(const hs_grammar *g, const uint8_t *text, int64_t len, int32_t *depths) {
    stk st = {0, 0, 0};
    int32_t cur = 0;
    int rc = HS_OK;
    if (!stk_push(&st, 0)) return HS_CAPACITY;
    for (int64_t i = 0; i <= len; i++) depths[i] = -1;
    depths[0] = 1;
    for (int64_t i = 0; i < len; i++) {
        rc = lex_byte(g, &cur, &st, text[i]);
        if (rc != HS_OK) break;
        depths[i + 1] = (int32_t)st.n;
    }
    free(st.s);
    return rc;
}
