/*
 * psc.h -- C ABI of the parser-stack-classification mask library (gfx950).
 *
 * Grammar-constrained decoding asks, at every decoding step and for every
 * sequence, which vocabulary tokens may follow the current prefix (the
 * constraint c(x), Sec. 2.1, eq. cons).  Parser stack classification
 * (Sec. 3) precomputes, once per (grammar, vocabulary) pair, one
 * deterministic automaton that reads the lexer state q and the parser stack
 * alpha top-first and lands in a state whose accepted vocabulary set is
 * precomputed (Sec. 3.5, eq. final_c and the sets A_s; Algorithm 1).  At
 * run time the automaton is walked once per sequence and the class's mask
 * is copied out (Algorithm 2, classification and mask steps); the mask is
 * then applied to the logits (Sec. 1, Fig. 1a).
 *
 * Conventions used by every call:
 *  - All sizes are element counts unless named *_bytes.
 *  - Masks are uint32 words, LSB-first: bit (v & 31) of word (v >> 5) is 1
 *    iff token v is allowed.  W = ceil(V / 32) words per row; bits >= V are 0.
 *  - Device pointers are HBM pointers owned by the caller; the library never
 *    frees them.  `stream` is a hipStream_t passed as void* (NULL = default
 *    stream).  Device calls only enqueue work; they never synchronise.
 *  - Every call returns psc_status; psc_last_error() gives a thread-local
 *    message for the last non-OK status.
 */
#ifndef PSC_H
#define PSC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PSC_OK = 0,
    PSC_E_INVALID_ARG = -1, /* null pointer, negative size, inconsistent shape */
    PSC_E_GRAMMAR = -2,     /* malformed tables (ids out of range, empty spelling, ...)
                               or grammar text (syntax, undefined symbol, ...)          */
    PSC_E_NOT_LALR1 = -3,   /* psc_grammar_compile: the grammar has LALR(1) conflicts  */
    PSC_E_OOM = -4,         /* host allocation failed (memory or threads)             */
    PSC_E_DEVICE = -5,      /* a HIP call or kernel launch failed                     */
    PSC_E_NOT_BOUND = -6,   /* device tables not bound (psc_bind_device)              */
    PSC_E_LIMIT = -7,       /* the construction exceeded a size limit                 */
    PSC_E_IO = -8,          /* a file could not be opened, read or written            */
    PSC_E_FORMAT = -9,      /* not a classifier file, unsupported version, corrupt or
                               inconsistent contents                                    */
    PSC_E_NOT_VIABLE = -10  /* psc_host_state: the text has a lexical or syntax error  */
} psc_status;

typedef enum { PSC_F32 = 0, PSC_BF16 = 1 } psc_dtype;

/*
 * The problem instance: the lexer T and the parser P that Algorithm 1 takes
 * as arguments (Sec. 2.2 FST, Sec. 2.4 PDA realised as LR tables, Sec. 4.1).
 * All arrays are host memory, row-major, read during psc_build only.
 *
 *  lex_next   [n_lex_states][256]  next lexer state on a byte, -1 = none.
 *                                  State 0 is q0 ("nothing pending").
 *  lex_accept [n_lex_states]       terminal the pending lexeme would be
 *                                  emitted as, -1 if not accepting.  Lexing is
 *                                  longest match with one byte of lookahead.
 *  terminal_ignored [n_terminals]  1 = consumed by the lexer, never parsed.
 *  end_terminal                    id of the end-of-input terminal $end.
 *  action [n_lr_states][n_terminals] (a & 3): 0 error, 1 shift to a >> 2,
 *                                  2 reduce by production a >> 2, 3 accept.
 *  goto_table [n_lr_states][n_nonterminals]  -1 = none.
 *  prod_lhs, prod_len [n_productions]        production 0 is the augmented
 *                                  start production.
 * Parser stacks are sequences of LR state ids (the stack alphabet Pi); LR
 * state 0 is the parser's start state, so the empty prefix has stack [0].
 */
typedef struct {
    int32_t n_lex_states;
    const int32_t *lex_next;
    const int32_t *lex_accept;
    int32_t n_terminals;
    const uint8_t *terminal_ignored;
    int32_t end_terminal;
    int32_t n_lr_states;
    int32_t n_nonterminals;
    const int32_t *action;
    const int32_t *goto_table;
    int32_t n_productions;
    const int32_t *prod_lhs;
    const int32_t *prod_len;
} psc_grammar;

/* The vocabulary V (Sec. 2.1): token v is bytes[offsets[v] .. offsets[v+1]).
 * Every spelling is non-empty except the EOS token's (eos_id, or -1 for
 * none).  Host memory, read during psc_build only. */
typedef struct {
    int32_t n_tokens;
    const uint8_t *bytes;
    const int64_t *offsets; /* [n_tokens + 1] */
    int32_t eos_id;
} psc_vocab;

typedef struct psc_handle psc_handle; /* opaque; owned by the library until psc_free */

typedef struct {
    int32_t vocab_size;        /* V                                           */
    int32_t mask_words;        /* W = ceil(V/32)                              */
    int32_t mask_stride_words; /* row stride of the device mask table (>= W)  */
    int32_t n_lex_states;      /* |Q|                                         */
    int32_t n_lr_states;       /* |Pi|                                        */
    int32_t n_classes;         /* distinct precomputed masks (rows)           */
    int64_t dfa_states_built;  /* automaton states before minimisation        */
    int32_t dfa_states;        /* after minimisation                          */
    int32_t dfa_rows;          /* states walked (not determined)              */
    int32_t dense_rows;        /* rows stored densely over Pi                 */
    int32_t max_sparse_edges;  /* largest sparse row                          */
    int64_t table_bytes;       /* classifier table bytes on the device        */
    int64_t mask_table_bytes;  /* mask table bytes on the device              */
    int64_t device_bytes;      /* total device buffer needed (psc_device_bytes) */
    double build_seconds;      /* wall time of psc_build                      */
    int32_t chain_states;      /* walked states stored as chain entries       */
    int32_t chains;            /* chains they form                            */
    int32_t mask_slices_unique; /* distinct 64-word slices of the mask rows   */
    int32_t bound_mask_layout; /* 0 unbound, PSC_BIND_FLAT or PSC_BIND_SLICED */
    int64_t sliced_mask_bytes; /* the mask table in the sliced layout: the
                                  distinct slices plus a slice id per row and
                                  slice (compare mask_table_bytes)            */
    int64_t skip_edges;        /* row entries that carry a skip over a run of
                                  wildcard chain states                       */
} psc_info_t;

/* Layouts of the mask table in the bound buffer (psc_bind_device_ex).
 *  PSC_BIND_FLAT    every class's row stored whole: one dependent load per
 *                   mask word after the class is known.
 *  PSC_BIND_SLICED  each row cut into 64-word slices and every distinct slice
 *                   stored once, with a slice id per (row, slice): the
 *                   runtime form of the precomputed masks compressed (the
 *                   paper's runtime mask memory, Tab. runtime_overhead), at
 *                   the cost of a second dependent load per mask word.
 * Every call gives bit-identical results under either layout. */
enum { PSC_BIND_FLAT = 1, PSC_BIND_SLICED = 2 };

/*
 * Offline construction (Algorithm 1; Sec. 3.1-3.5), CPU only.  Lexes every
 * token from every lexer state (R_q(v), Sec. 3.1), simulates the parser on
 * every realizable terminal sequence against a stack read lazily top-first
 * (the transducers P_eps, P~_a and P_w of Sec. 3.3-3.4, run in lock step),
 * determinises the union over (q, v) into one automaton (eq. final_c),
 * minimises it, deduplicates the per-state accepted sets A_s into classes,
 * and flattens everything into device-ready arrays.
 * On success *out receives a new handle.  Errors: PSC_E_INVALID_ARG (null
 * pointers, sizes <= 0), PSC_E_GRAMMAR (ids out of range, a non-EOS token with
 * an empty spelling), PSC_E_OOM, PSC_E_LIMIT (more subset states built, over
 * all lexer states and before minimisation, than the environment variable
 * PSC_BUILD_MAX_STATES allows; default 10^9).  The construction runs on as
 * many threads as the process's CPU affinity mask holds, at most
 * OMP_NUM_THREADS when that is set and at most 32; PSC_BUILD_THREADS
 * overrides.
 */
psc_status psc_build(const psc_grammar *grammar, const psc_vocab *vocab, psc_handle **out);

/*
 * Grammar text -> the tables psc_build takes (T and P, the arguments of
 * Algorithm 1; Sec. 4.1 obtains P from an LALR(1) generator).  One statement
 * per line, '#' starts a comment outside quotes and slashes:
 *   %start NAME                the start nonterminal
 *   %ignore NAME /regex/       a terminal the lexer consumes and drops
 *   %literal "text" [PRIO]     declare a literal terminal at this point
 *   NAME[.PRIO]: /regex/       a regex terminal
 *   name: item item | item     productions of `name`; an item is a declared
 *                              terminal, a "literal" (declared on first use)
 *                              or a nonterminal; '|' separates alternatives,
 *                              an empty one is the empty production, and a
 *                              line starting with '|' continues the rule.
 * Literals take \\ \" \n \t \r \xHH.  Regexes are over bytes: . [...] [^...]
 * ( ) (?: ) | * + ? {m} {m,} {m,n} and \n \t \r \f \v \0 \xHH \d \w \s;
 * another escaped byte stands for itself (\/ is a slash).
 * Lexing is longest match with one byte of lookahead; a tie on the same
 * lexeme goes to the higher priority, then a literal over a regex, then the
 * earlier declaration.  Terminal ids follow declaration order, then $END;
 * nonterminal ids follow first appearance as a left side, then $start;
 * production 0 is $start -> start.  The LR(1) tables are LALR(1), built from
 * the LR(0) automaton with DeRemer-Pennello lookaheads; nothing is resolved
 * by precedence and no reduction is defaulted.
 * On success *out owns the tables (psc_grammar_free).  Errors:
 * PSC_E_INVALID_ARG, PSC_E_GRAMMAR (syntax, undefined or misused symbol, a
 * terminal matching the empty string; the message names the line),
 * PSC_E_NOT_LALR1 (the message names the first conflicts: state, terminal
 * and the two actions), PSC_E_LIMIT (the terminals' NFA over 4,000,000
 * states, the lexer DFA over 1,000,000 before minimisation, or its subsets
 * holding over 200,000,000 NFA states in all; groups nested deeper than 500
 * or more than 500 repetition operators in a row are PSC_E_GRAMMAR),
 * PSC_E_OOM.
 */
typedef struct psc_compiled_grammar psc_compiled_grammar;
psc_status psc_grammar_compile(const char *text, size_t len, psc_compiled_grammar **out);
/* The tables as the psc_grammar that psc_build takes; the pointers stay valid
 * until psc_grammar_free. */
psc_status psc_grammar_view(const psc_compiled_grammar *g, psc_grammar *out);
/* Name of terminal id (terminal != 0) or nonterminal id; NULL out of range. */
const char *psc_grammar_symbol_name(const psc_compiled_grammar *g, int32_t terminal, int32_t id);
void psc_grammar_free(psc_compiled_grammar *g);
/* psc_grammar_compile, then psc_build on the result. */
psc_status psc_build_from_text(const char *text, size_t len, const psc_vocab *vocab, psc_handle **out);

/*
 * Persistence of a built classifier, so that Algorithm 1 runs once per
 * (grammar, vocabulary) pair (the preprocessing the paper stores, Sec. 4 /
 * Tab. preprocess).  psc_save writes everything a handle holds (classifier
 * table, mask table, and the lexer, parser and vocabulary psc_advance reads)
 * to `path`, each part checksummed, the large ones deflate-compressed.
 * psc_load reads such a file into a new, unbound handle.  A loaded file is
 * untrusted: psc_load verifies the checksums and the structure the device
 * kernels rely on (every ref names a row, a chain entry of the right kind or
 * a class; chains end within one wavefront load; the lexer, parser and
 * vocabulary pass psc_build's input checks) before it returns a handle.
 * Files are little-endian and tied to this library's format version.
 * Errors: PSC_E_INVALID_ARG, PSC_E_IO, PSC_E_FORMAT, PSC_E_OOM.
 */
psc_status psc_save(const psc_handle *h, const char *path);
psc_status psc_load(const char *path, psc_handle **out);

/* Sizes and statistics of a built handle. */
psc_status psc_info(const psc_handle *h, psc_info_t *out);

/* Device bytes psc_bind_device needs (256-byte aligned buffer). */
size_t psc_device_bytes(const psc_handle *h);

/* Device bytes psc_bind_device_ex needs for the mask layout in `flags`
 * (PSC_BIND_FLAT, PSC_BIND_SLICED, or 0 for the default layout). */
size_t psc_device_bytes_ex(const psc_handle *h, uint32_t flags);

/*
 * Copy the classifier and mask tables, and the lexer, parser and vocabulary
 * that psc_advance reads, into caller-allocated device memory (dev_buf,
 * nbytes >= psc_device_bytes, 256-byte aligned) on `stream`, and zero the
 * device error counter.  The buffer must stay alive and unmodified
 * while the handle is used; the handle keeps only the pointer.  Rebinding
 * replaces the previous binding.  Errors: PSC_E_INVALID_ARG, PSC_E_DEVICE,
 * PSC_E_OOM (the tables derived at bind time do not fit in host memory).
 */
psc_status psc_bind_device(psc_handle *h, void *dev_buf, size_t nbytes, void *stream);

/* psc_bind_device with the mask table in the layout `flags` selects
 * (PSC_BIND_FLAT or PSC_BIND_SLICED; 0 = the default, PSC_BIND_FLAT);
 * nbytes >= psc_device_bytes_ex(h, flags).  Also clears the class predictor
 * (psc_predictor_fill) and the device counters. */
psc_status psc_bind_device_ex(psc_handle *h, void *dev_buf, size_t nbytes, uint32_t flags, void *stream);

/*
 * Per-step mask computation (Algorithm 2, classification and mask steps).
 * For every sequence b < B: start from the automaton state for
 * lexer_states[b], read its stack top-first, stop early once the class is
 * determined, and copy that class's precomputed mask into
 * out_bitmask[b][0..W).
 *  stacks       device int32, the B stacks concatenated in batch order, each
 *               stored bottom -> top (LR start state first, top last); the
 *               total may exceed 2^31 symbols.  Each sequence finds its
 *               stack by summing the lengths before it (O(B) reads per
 *               sequence): for large batches the dense layout below is
 *               cheaper.
 *  stack_lens   device int32 [B], each >= 1 (a negative length holds no
 *               symbols of `stacks`).
 *  lexer_states device int32 [B].
 *  out_bitmask  device uint32 [B][W], W = ceil(V/32), fully written.
 * A sequence with an out-of-range lexer state or stack symbol, or a length
 * <= 0, gets an all-zero row and increments the device error counter; a
 * well-formed stack that no prefix can produce gives an unspecified row.
 * B == 0 is a no-op.  Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND, PSC_E_DEVICE.
 */
psc_status psc_compute_masks(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                             const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask,
                             void *stream);

/*
 * The ragged-stack calls (psc_compute_masks, psc_compute_classes,
 * psc_compute_and_apply, psc_compute_and_argmax) trust the device lengths to
 * fit `stacks`.  Their *_n forms take n_stack, the number of int32 symbols
 * the caller's `stacks` buffer holds (>= 0): a sequence whose stack would
 * reach past it (offset + length > n_stack) is a rejected input (all-zero
 * row, or -1, and a count in the error counter) and is never read.
 * Otherwise identical to the calls without _n.
 */
psc_status psc_compute_masks_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                               const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                               uint32_t *out_bitmask, void *stream);

/*
 * Mask application (Sec. 1, Fig. 1a: logits are masked before sampling), in
 * place on a contiguous device tensor logits[B][V] of `dtype`:
 *   logits[b][v] = -inf   wherever bit v of bitmask[b] (uint32 [B][ceil(V/32)]) is 0;
 * allowed entries are left untouched (their bits, NaN payloads included, do
 * not change).  B == 0 or V == 0 is a no-op.  Errors: PSC_E_INVALID_ARG,
 * PSC_E_DEVICE.
 */
psc_status psc_apply_mask(void *logits, psc_dtype dtype, const uint32_t *bitmask, int32_t B,
                          int32_t V, void *stream);

/*
 * The classification step of Algorithm 2 alone: out_classes[b] = the class
 * of sequence b, i.e. the row of the precomputed mask table that
 * psc_compute_masks would copy (psc_class_mask_host returns that row on the
 * host).  Inputs as for psc_compute_masks; out_classes is device int32 [B].
 * An out-of-range input gives -1 and increments the device error counter.
 * For callers that share or cache masks by class, and to time the walk on
 * its own.  B == 0 is a no-op.  Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND,
 * PSC_E_DEVICE.
 */
psc_status psc_compute_classes(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                               const int32_t *lexer_states, int32_t B, int32_t *out_classes, void *stream);
psc_status psc_compute_classes_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                 const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                 int32_t *out_classes, void *stream);

/*
 * The whole per-step path in one launch: psc_compute_masks followed by
 * psc_apply_mask (Algorithm 2, classification and mask steps; Sec. 1,
 * Fig. 1a), fused so that each workgroup walks its sequence, gathers its
 * slice of the class's mask row and applies it to the logits directly.
 *  stacks, stack_lens, lexer_states  as for psc_compute_masks.
 *  out_bitmask  device uint32 [B][W], fully written as by psc_compute_masks;
 *               may be NULL when only the masked logits are wanted.
 *  logits       device, contiguous [B][V] of `dtype`, masked in place as by
 *               psc_apply_mask; V must equal the vocabulary size of `h`.
 * A rejected sequence (see psc_compute_masks) gets an all-zero mask row, so
 * its whole logits row becomes -inf, and counts once in the error counter.
 * Results are bit-identical to the two separate calls.  B == 0 is a no-op.
 * Errors: PSC_E_INVALID_ARG (also V != vocabulary size), PSC_E_NOT_BOUND,
 * PSC_E_DEVICE.
 */
psc_status psc_compute_and_apply(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                 const int32_t *lexer_states, int32_t B, uint32_t *out_bitmask, void *logits,
                                 psc_dtype dtype, int32_t V, void *stream);
psc_status psc_compute_and_apply_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                   const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                   uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                   void *stream);

/*
 * The class predictor.  A walk's first step from start[q] leaves the start
 * block of lexer state q in one of a few ways (which edge, or how far along
 * a chain); psc_compute_and_apply, psc_compute_masks and psc_compute_classes
 * record, per such (q, way), the class the walk then reached.  When a later
 * walk leaves the same way, the workgroups of psc_compute_and_apply and
 * psc_compute_masks start loading that class's mask words (and the logits it
 * leaves partly allowed) while the walk goes on, and use them if the walk
 * ends in that class; otherwise they load the right ones.  The predictor
 * only decides what is loaded early, never a result: every output is the
 * same whatever it holds.  It lives in the bound buffer; concurrent calls on
 * one handle may overwrite each other's entries, which is harmless.
 * psc_compute_classes over sample prefix states (e.g. a prompt set) fills it
 * before decoding starts.
 *
 * psc_predictor_fill sets every entry to `cls` (-1: no prediction; else a
 * class id < n_classes), on `stream`.  psc_predictor_updates reads
 * (synchronously) the number of entries the calls above have changed since
 * the last reset, i.e. walks whose class differed from the prediction, and
 * optionally resets it.  Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND,
 * PSC_E_DEVICE.
 */
psc_status psc_predictor_fill(const psc_handle *h, int32_t cls, void *stream);

/*
 * Options of a handle's device calls (a bitwise OR; 0 = the defaults):
 *  PSC_OPT_SPECULATE  psc_compute_and_apply loads the predicted class's mask
 *                     words and partly allowed logits during the walk (the
 *                     class predictor above); results are identical either
 *                     way.  Off by default: on MI355X the walk's loads and
 *                     the workgroup's second barrier cost about what the
 *                     early loads save.
 * Errors: PSC_E_INVALID_ARG (null handle, unknown option).
 */
enum { PSC_OPT_SPECULATE = 1 };
psc_status psc_set_options(psc_handle *h, uint32_t options);
psc_status psc_predictor_updates(const psc_handle *h, uint32_t *out, int32_t reset, void *stream);

/*
 * psc_compute_and_apply_n with a per-wavefront timeline for profiling: every
 * wavefront of the launch writes one record of four uint64 to `records`
 * (device memory, n_records >= psc_timeline_records(h, B, dtype)), in the
 * order (sequence, slice, wavefront).  Times are ticks of the GPU's constant
 * 100 MHz clock:
 *   [0] its start;
 *   [1] (after the walk's first step, with PSC_OPT_SPECULATE; else = start)
 *       - start, then (its class known) - start << 32;
 *   [2] (its last store issued) - start, then, << 32: wavefront | XCD << 3 |
 *       prediction held << 7 | class known at the first step << 8;
 *   [3] sequence | slice << 32.
 * Results are those of psc_compute_and_apply_n.  Fast path only
 * (V % 32 == 0, 16-byte aligned logits): PSC_E_INVALID_ARG otherwise.
 */
int64_t psc_timeline_records(const psc_handle *h, int32_t B, psc_dtype dtype);
psc_status psc_compute_and_apply_timeline(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                          const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                          uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                          uint64_t *records, int64_t n_records, void *stream);

/*
 * Greedy decoding folded into the mask step (the mask decides which logits
 * sampling may see, Sec. 1 / Fig. 1a): for every sequence, the walk and then
 *   out_tokens[b] = argmax over allowed tokens v of logits[b][v]
 * (device int32 [B]): ties go to the lowest id, a NaN logit counts above
 * every number, -0 equals +0, and a row with no allowed token (or a rejected
 * input, as in psc_compute_masks) gives -1.  The logits (device, contiguous
 * [B][V] of `dtype`, V = the vocabulary size) are only read, and only the
 * 16-byte groups that hold an allowed token.  One kernel launch; the
 * workgroups of a sequence combine their results in a per-sequence slot and
 * arrival counter of the bound device buffer, which each call leaves at
 * zero, so argmax calls on one handle must not overlap in time (one stream,
 * or synchronised streams).  B <= 65535.  Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND, PSC_E_DEVICE.
 */
psc_status psc_compute_and_argmax(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                                  const int32_t *lexer_states, int32_t B, const void *logits, psc_dtype dtype,
                                  int32_t V, int32_t *out_tokens, void *stream);
psc_status psc_compute_and_argmax_n(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                    const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                    const void *logits, psc_dtype dtype, int32_t V, int32_t *out_tokens,
                                    void *stream);

/*
 * Device-resident prefix states (Sec. 3.2: a prefix is represented by its
 * lexer state and parser stack; Algorithm 2 lexes and parses each new token
 * before classifying).  B sequences keep their states in HBM between decoding
 * steps, in a dense layout:
 *  stacks        device int32 [B][cap]; stack b is stacks[b*cap .. b*cap +
 *                stack_lens[b]), bottom first (LR state 0, the parser's start
 *                state, at the bottom), top last.
 *  stack_lens    device int32 [B], 1 <= stack_lens[b] <= cap.
 *  lexer_states  device int32 [B].
 * All three are caller-owned and updated in place by psc_state_reset and
 * psc_advance; the masks of the states are computed by the *_dense calls.
 */

/* Status per sequence written by psc_advance. */
enum {
    PSC_ADV_OK = 0,        /* advanced: the new state is in place                          */
    PSC_ADV_REJECTED = 1,  /* the lexer has no move or an emitted terminal is not shifted;
                              state unchanged                                             */
    PSC_ADV_EOS = 2,       /* EOS and the prefix is a sentence of the language; unchanged  */
    PSC_ADV_OVERFLOW = 3,  /* the new stack would not fit cap, or the token pushes more
                              than 192 states above what it keeps; unchanged              */
    PSC_ADV_BAD_INPUT = 4, /* token, length, lexer state or a stack symbol the token's
                              parsing reads out of range; unchanged                       */
    PSC_ADV_SKIPPED = 5    /* tokens[b] < 0: nothing to do                                 */
};

/* Every sequence to the empty prefix: lexer state 0 (q0), stack [0].
 * Errors: PSC_E_INVALID_ARG, PSC_E_DEVICE. */
psc_status psc_state_reset(const psc_handle *h, int32_t *stacks, int32_t cap, int32_t *stack_lens,
                           int32_t *lexer_states, int32_t B, void *stream);

/*
 * Advance every sequence b by token tokens[b] (device int32 [B]; < 0 = skip),
 * the lexing and parsing steps of Algorithm 2 (Sec. 3.2): the token's bytes
 * are lexed from the lexer state (longest match, one byte of lookahead), every
 * terminal a finished lexeme yields is fed to the LR parser (its reductions,
 * then a shift), and the lexeme still pending after the last byte stays in
 * the lexer state.  EOS instead checks that the prefix is a sentence.  Writes
 * status[b] (device int32 [B], PSC_ADV_*); the state changes only with
 * PSC_ADV_OK.  It does not look ahead: a token can be advanced over and leave
 * a pending lexeme that nothing can complete -- the next mask is then all
 * zero (the masks reject such tokens beforehand).  Errors: PSC_E_INVALID_ARG,
 * PSC_E_NOT_BOUND, PSC_E_DEVICE.
 */
psc_status psc_advance(const psc_handle *h, int32_t *stacks, int32_t cap, int32_t *stack_lens,
                       int32_t *lexer_states, int32_t B, const int32_t *tokens, int32_t *status, void *stream);

/* psc_compute_masks on device-resident states (dense layout above); a
 * length outside [1, cap] is a rejected input. */
psc_status psc_compute_masks_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                   const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                   uint32_t *out_bitmask, void *stream);

/* psc_compute_classes on device-resident states (dense layout above). */
psc_status psc_compute_classes_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                     const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                     int32_t *out_classes, void *stream);

/* psc_compute_and_apply on device-resident states (dense layout above). */
psc_status psc_compute_and_apply_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                       const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                       uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V,
                                       void *stream);

/*
 * One whole decoding step of Algorithm 2 in one launch (two when the batch
 * is too large for all its workgroups to run at once), on device-resident
 * states: the lexing and parsing steps (psc_advance by tokens[b]), then the
 * classification and mask steps of the new state, applied to the logits
 * (psc_compute_and_apply_dense).  The results (new states, status, bitmask,
 * masked logits, error counter) are bit-identical to copying each state to
 * the output buffers, calling psc_advance on them, then
 * psc_compute_and_apply_dense.
 *  stacks_in, lens_in, qs_in     device, the current states (dense layout
 *                                above, `cap`); only read.
 *  stacks_out, lens_out, qs_out  device, the same shapes: receive the new
 *                                states (a state that does not advance is
 *                                copied unchanged).  They must not overlap the
 *                                inputs (checked): every workgroup of a
 *                                sequence reads the old state while one writes
 *                                the new one, so callers alternate two buffers.
 *  tokens, status                as for psc_advance.
 *  out_bitmask, logits, dtype, V as for psc_compute_and_apply.
 * B == 0 is a no-op.  Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND,
 * PSC_E_DEVICE.
 */
psc_status psc_decode_step(const psc_handle *h, const int32_t *stacks_in, const int32_t *lens_in,
                           const int32_t *qs_in, int32_t *stacks_out, int32_t *lens_out, int32_t *qs_out,
                           int32_t cap, int32_t B, const int32_t *tokens, int32_t *status,
                           uint32_t *out_bitmask, void *logits, psc_dtype dtype, int32_t V, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * results as psc_compute_and_argmax_n, with the per-sequence argmax records
 * in a fixed array of the library's own (one copy per GPU, 512 KiB, taken
 * and cleared by the first psc_bind_device on that GPU and held until the
 * process ends) instead of the bound buffer.  The call allocates nothing.
 * B <= 4096, else PSC_E_INVALID_ARG.  Every call on one GPU shares that
 * GPU's array (through any handle): calls that overlap in time on one GPU
 * race and give wrong tokens; each completed call leaves the array zeroed.
 * Errors: PSC_E_INVALID_ARG, PSC_E_NOT_BOUND, PSC_E_DEVICE.
 */
psc_status psc_compute_and_argmax_noalloc(const psc_handle *h, const int32_t *stacks, int64_t n_stack,
                                          const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                          const void *logits, psc_dtype dtype, int32_t V, int32_t *out_tokens,
                                          void *stream);

/* psc_compute_and_argmax on device-resident states (dense layout above). */
psc_status psc_compute_and_argmax_dense(const psc_handle *h, const int32_t *stacks, int32_t cap,
                                        const int32_t *stack_lens, const int32_t *lexer_states, int32_t B,
                                        const void *logits, psc_dtype dtype, int32_t V, int32_t *out_tokens,
                                        void *stream);

/* Read (synchronously, on `stream`) and optionally reset the device counter
 * of sequences that psc_compute_masks rejected as out of range. */
psc_status psc_device_error_count(const psc_handle *h, uint32_t *out, int32_t reset, void *stream);

/*
 * Host walk of the same automaton, for triage and for timing the method on
 * one CPU thread as the paper does: classes for B host-resident prefix
 * states (same stack layout as psc_compute_masks, host pointers).  It is not
 * used by any device call.  out_classes[b] = -1 for an out-of-range input.
 */
psc_status psc_classify_host(const psc_handle *h, const int32_t *stacks, const int32_t *stack_lens,
                             const int32_t *lexer_states, int32_t B, int32_t *out_classes);

/* Copy class c's mask row (W words) to host memory. */
psc_status psc_class_mask_host(const psc_handle *h, int32_t cls, uint32_t *out_row);

/*
 * The prefix state of a text (Sec. 3.2: the lexer state plus the LR parser
 * stack after the text), computed on the host from the handle's lexer and
 * parser tables, for callers that start decoding from a prompt or a partial
 * output: its (q, stack) is what psc_compute_masks and the device states
 * take.  The text (`len` bytes, host memory) is lexed from q0 by longest
 * match with one byte of lookahead; every finished lexeme whose terminal is
 * not ignored is fed to the parser (its reductions, then its shift); the
 * last lexeme stays pending in *q.  The stack, s0 first, goes to `stack`
 * (cap int32, host memory), its length to *stack_len.  Whether the pending
 * lexeme can still complete is not checked: that is what the mask answers.
 * Errors: PSC_E_INVALID_ARG (null pointers, cap < 1), PSC_E_NOT_VIABLE (a
 * byte that no lexeme can take, or a terminal the parser rejects; the
 * outputs are then unspecified), PSC_E_LIMIT (the stack would exceed cap),
 * PSC_E_GRAMMAR (reductions that never end, only on corrupt tables).  Not
 * used by any device call.
 */
psc_status psc_host_state(const psc_handle *h, const uint8_t *text, size_t len, int32_t *q, int32_t *stack,
                          int32_t cap, int32_t *stack_len);

/* Release the handle and its host tables (never the caller's device buffer). */
void psc_free(psc_handle *h);

/* Thread-local message for the last non-OK status of this thread. */
const char *psc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* PSC_H */
