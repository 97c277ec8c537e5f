/* epic.h - C ABI of the MI355X (gfx950) validity-check hot path of EPIC
 * (Efficient and Parallel Inference under CFG constraints, arxiv 2606.00722).
 *
 * Per denoising step a diffusion LM proposes (position, token) commits for a
 * batch of partially masked token sequences.  This library decides, for every
 * proposal, whether the sequence stays completable under a context-free
 * grammar (Sec. 3: Valid_G(x, D) = 1[L(G) cap C_{x+D} != empty], masked runs
 * read as Sigma*), and then chooses the relaxed compatible subset of the
 * valid proposals to commit together (Sec. 4.3, Alg. 4).
 *
 * Conventions for every call:
 *  - Pointers named d_* are device pointers (HIP device memory, e.g. PyTorch
 *    tensors); all other pointers are host pointers.  Host data is copied
 *    before the call returns; the caller keeps ownership of everything it
 *    passes in.
 *  - Device work is enqueued on `stream` and the call returns without
 *    waiting; outputs are valid after the stream is synchronised.
 *  - A context is used by one host thread at a time; distinct contexts are
 *    independent.  Calls on one context that overlap on different streams
 *    must not share a workspace.
 *  - Errors detectable on the host are returned immediately as a negative
 *    epic_status and nothing is enqueued.  Errors that only the device can
 *    see mark the affected candidate (verdict 2) and set a sticky device flag
 *    that epic_ctx_device_error() reads after synchronising.
 */
#ifndef EPIC_H
#define EPIC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EPIC_OK = 0,
  EPIC_ERR_NULL = -1,        /* a required pointer is NULL */
  EPIC_ERR_ARG = -2,         /* a size or index argument is out of range */
  EPIC_ERR_CAPACITY = -3,    /* larger than the context or workspace was sized for */
  EPIC_ERR_LEXER = -4,       /* lexer DFA malformed (start accepts, not trim, bad label) */
  EPIC_ERR_GRAMMAR = -5,     /* undefined symbol, start not a nonterminal, too large */
  EPIC_ERR_VOCAB = -6,       /* token empty or longer than 8 bytes */
  EPIC_ERR_HIP = -7,         /* a HIP runtime call failed */
  EPIC_ERR_STATE = -8,       /* memo not built yet */
  EPIC_ERR_UNSUPPORTED = -9  /* outside the sizes the library supports (see below) */
} epic_status;

/* Device-side sticky error bits, read by epic_ctx_device_error(). */
#define EPIC_DEV_BAD_CANDIDATE 1u  /* position not masked, token/sequence/position out of range */
#define EPIC_DEV_CAPACITY 2u       /* a chart or graph buffer overflowed: verdict 2 written */
#define EPIC_DEV_BAD_SELECT 4u     /* duplicate positions or NaN confidence among valid candidates */
/* With EPIC_DEV_CAPACITY, bit 8+i names the buffer that overflowed: i = 1 chart
 * slots of one row, 2 slot hash, 3 row tasks, 4 chart entries, 5 graph nodes,
 * 6 in-edges of a node, 7 frontier, 8 emission events. */

typedef struct epic_ctx epic_ctx;

/* Lexer DFA: the compiled lexical map (Alg. 1 "compile the lexical map").
 * States 0..num_states-1, state 0 is the start state and must not accept;
 * every state must reach an accepting state (trim).  trans[q*256 + byte] is
 * the successor or -1.  accept[q] is -1 (not accepting), -2 (a skip lexeme
 * such as whitespace) or a grammar terminal id.  Lexing is greedy with one
 * byte of lookahead and no backtracking: a lexeme ends when the next byte has
 * no transition; the earlier-listed rule already decided the label.
 * Supported: num_states <= 256. */
typedef struct {
  int32_t num_states;
  const int16_t* trans;
  const int16_t* accept;
} epic_lexer_desc;

/* Grammar G = (V, Sigma_lex, P, S) (Sec. 3).  Terminals are 0..T-1,
 * nonterminals T..T+N-1; production p is lhs[p] -> rhs[rhs_offsets[p] ..
 * rhs_offsets[p+1]).  Empty right-hand sides are allowed.
 * Supported: T <= 63, N <= 64, at most 512 dotted items (sum of |rhs|+1,
 * plus two for the augmented start production). */
typedef struct {
  int32_t num_terminals, num_nonterminals, start, num_productions;
  const int32_t* lhs;
  const int32_t* rhs_offsets;
  const int32_t* rhs;
} epic_grammar_desc;

/* Tokenizer vocabulary Gamma: token t has bytes[offsets[t] .. offsets[t+1]),
 * 1 to 8 bytes. */
typedef struct {
  int32_t vocab_size;
  const uint8_t* bytes;
  const int32_t* offsets;
} epic_vocab_desc;

/* Create a context: validates the descriptors, builds the constant tables
 * (dotted items, prediction closure, the lexer's gap automaton reduced to its
 * left-language classes, the regular cover of App. A.2), uploads them and
 * allocates the memo table (vocab_size * num_states * 16 bytes).  max_batch,
 * max_seq_len and max_cands bound later calls (max_seq_len <= 1024).
 * *out receives the context. */
epic_status epic_ctx_create(const epic_lexer_desc* lexer, const epic_grammar_desc* grammar,
                            const epic_vocab_desc* vocab, int32_t max_batch, int32_t max_seq_len,
                            int32_t max_cands, epic_ctx** out);

void epic_ctx_destroy(epic_ctx* ctx);

/* Bytes of device workspace that epic_validate_batch,
 * epic_select_compatible and epic_commit_fallback need (the caller allocates
 * it, 256-byte aligned, and zeroes it once after allocating it).
 * Besides per-call scratch the workspace keeps, between calls, the recorded
 * walks of each sequence (its chart state at every masked run, tagged with the
 * context and the sequence walked).  A later call on the same context and
 * workspace resumes a sequence's walk at the last recorded masked run that
 * starts at or before the first token that changed.  Records of another
 * context (other tables, another process, or a context since destroyed) fail
 * the tag check and the sequence is walked from the start, as in a zeroed
 * workspace.  The tag covers the record headers, not the chart storage they
 * point into, so the caller must zero a newly allocated workspace (memory
 * that held this context's earlier workspace could otherwise carry valid
 * headers over overwritten charts) and must not modify it between calls;
 * under these two rules results do not depend on its contents, only the time
 * taken does. */
size_t epic_workspace_bytes(const epic_ctx* ctx);

/* Number of graph nodes one masked run contributes: the left-language
 * classes of the lexer's gap automaton (diagnostics; 2 for lexers whose
 * whitespace can separate any two lexemes: inside whitespace, and after
 * anything else). */
int32_t epic_gap_classes(const epic_ctx* ctx);

/* Number of 32-bit words of an item bitset (diagnostics; the productions'
 * dotted items packed so that none straddles a word, rounded up to a power
 * of two; each chart entry stores this many words). */
int32_t epic_item_words(const epic_ctx* ctx);

/* Alg. 2, lexing memoization: for every token t and lexer state q the greedy
 * lexing of t's bytes from q, without a final flush, into the context's memo
 * table.  Entry (t, q) sits at byte offset (t*num_states + q)*16:
 *   [0..1] state after the token (little-endian u16, 0xFFFF = the lexer dies)
 *   [2]    number of emissions (skip lexemes included)
 *   [3]    emission mask: bit j set when reading byte j ended a lexeme
 *   [4..11] emitted labels in order (terminal id, 0xFF = skip), unused = 0
 *   [12..15] zero.  A dead entry is all zero except bytes 0..1.
 * Enqueued on `stream`; must complete before validation reads the memo. */
epic_status epic_lexmemo_build(epic_ctx* ctx, hipStream_t stream);

/* Copy the memo table to host memory (bytes >= vocab_size*num_states*16).
 * Synchronous. */
epic_status epic_memo_export(const epic_ctx* ctx, void* host_dst, size_t bytes);

/* Validity of each proposal (Sec. 3 Valid; Alg. 3 is the recogniser):
 * verdict[c] = Valid_G(x_b, {(pos[c], tok[c])}) for b = cand_seq[c], i.e. 1
 * if x_b with token tok[c] at position pos[c] can still be completed into a
 * sentence of L(G), else 0; 2 if the candidate is malformed (sequence or
 * position out of range, position not masked in x_b, token out of range).
 * d_seqs: int32 [B*n] row-major, -1 = MASK.  d_cand_*: int32 [C].
 * d_verdict: uint8 [C].  Every candidate is judged against the same x_b.
 * d_workspace: at least epic_workspace_bytes(ctx) bytes. */
epic_status epic_validate_batch(epic_ctx* ctx, const int32_t* d_seqs, int32_t B, int32_t n,
                                const int32_t* d_cand_seq, const int32_t* d_cand_pos,
                                const int32_t* d_cand_tok, int32_t C, uint8_t* d_verdict,
                                void* d_workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that must not allocate, harnesses that forbid
 * hipMalloc): epic_validate_batch without a workspace.  The verdicts are
 * epic_validate_batch's.  The walks keep their charts in a scratch array of
 * 256 MiB that the library holds in device memory, one per GPU, from the
 * first context created on that GPU until the process ends; the call itself
 * calls no hipMalloc, hipFree or other allocating routine.  Every call on a
 * GPU shares that GPU's array, so calls that overlap on one GPU (other
 * streams, contexts or host threads) race: the caller serialises them.
 * Nothing in the array must start at zero (a walk writes every chart row
 * before reading it, and nothing is kept between calls: no prefix sharing,
 * no walk records).  As many walks run at once as chart slots of the
 * context fit in the array (at most 1024); EPIC_ERR_CAPACITY when not even
 * one fits (the slot size grows with the context's max_seq_len and item
 * words: about 11 MB for 16-word items at 256 or more tokens). */
epic_status epic_validate_batch_noalloc(epic_ctx* ctx, const int32_t* d_seqs, int32_t B, int32_t n,
                                        const int32_t* d_cand_seq, const int32_t* d_cand_pos,
                                        const int32_t* d_cand_tok, int32_t C, uint8_t* d_verdict,
                                        hipStream_t stream);

/* Relaxed compatible-subset selection (Alg. 4): per sequence, the candidates
 * with verdict 1 are sorted by descending confidence (float32, ties to the
 * lower candidate index) and passed to RelaxedSelect followed by
 * ExactShrink; halves put the first ceil(|C|/2) candidates on the
 * high-confidence side.  The relaxed check is the emptiness test of the
 * regular cover intersected with the completion automaton (App. A.2);
 * the exact check is Valid.  d_selected: uint8 [C], 1 = in the returned
 * subset B (empty, or at least two candidates whose joint application is
 * exactly valid).  A sequence whose verdict-1 candidates repeat a position or
 * carry a NaN confidence selects nothing and sets EPIC_DEV_BAD_SELECT; one
 * with more than 64 verdict-1 candidates selects nothing and sets
 * EPIC_DEV_CAPACITY; a verdict-1 candidate that is not a legal update sets
 * EPIC_DEV_BAD_CANDIDATE.
 * d_counts (optional, device int64 [2]) accumulates the number of cover and
 * exact checks Alg. 4 calls.  Some calls are answered without a walk: a
 * repeated check, or one an answered check decides (a pass carries to
 * subsets, a failure to supersets, an exact pass to the cover check, a cover
 * failure to the exact check); the answer is the one the walk would give. */
epic_status epic_select_compatible(epic_ctx* ctx, const int32_t* d_seqs, int32_t B, int32_t n,
                                   const int32_t* d_cand_seq, const int32_t* d_cand_pos,
                                   const int32_t* d_cand_tok, const float* d_conf,
                                   const uint8_t* d_verdict, int32_t C, uint8_t* d_selected,
                                   int64_t* d_counts, void* d_workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/* The sequential fallback that follows the relaxed batch in EPIC decoding
 * (App. C.1: Alg. 1 and the paragraph after it): per sequence b,
 * with the selected set B (d_selected, as written by epic_select_compatible)
 * committed to x_b, the other candidates of b are taken by descending
 * confidence (float32, ties to the lower candidate index); each is committed
 * when x_b + (everything committed so far) + c is valid (Sec. 3 Valid), until
 * d_num_commit[b] - |B| more are committed (n_t of the step) or the
 * candidates run out.  Candidates with verdict != 1 are never committed: a
 * candidate invalid on x_b stays invalid once more masked positions are
 * filled.  d_num_commit: device int32 [B].  d_accepted: uint8 [C], 1 = the
 * fallback committed the candidate (B's candidates and the others 0); the
 * caller applies B and the accepted candidates to x.  Inputs are not
 * modified.  The same input rules as epic_select_compatible apply: a sequence
 * whose verdict-1 candidates repeat a position or carry a NaN confidence, or
 * number more than 64, commits nothing and sets the corresponding flag. */
epic_status epic_commit_fallback(epic_ctx* ctx, const int32_t* d_seqs, int32_t B, int32_t n,
                                 const int32_t* d_cand_seq, const int32_t* d_cand_pos, const int32_t* d_cand_tok,
                                 const float* d_conf, const uint8_t* d_verdict, const uint8_t* d_selected,
                                 const int32_t* d_num_commit, int32_t C, uint8_t* d_accepted, void* d_workspace,
                                 size_t workspace_bytes, hipStream_t stream);

/* Synchronise `stream`, then read and clear the sticky device error bits
 * (EPIC_DEV_*) into *flags. */
epic_status epic_ctx_device_error(epic_ctx* ctx, hipStream_t stream, uint32_t* flags);

/* Diagnostics: synchronise `stream`, then read and clear the work counters
 * accumulated by all walks since the last call: out[0] graph walks (one per
 * validity or cover check), out[1] chart entries written (origin slots of
 * Earley rows: 4*W bytes of items for W item words, an 8-byte summary of the
 * expected nonterminals and a 2-byte origin), out[2] memo entries read (16
 * bytes each), out[3] graph nodes built, out[4] chart entries examined by
 * completion and scan steps (summary and origin read), out[5] of those,
 * entries whose items were read. */
epic_status epic_ctx_work_counters(epic_ctx* ctx, hipStream_t stream, int64_t* out);

/* Diagnostics: per-kernel timing.  With enable != 0, every kernel the
 * context launches from then on is bracketed by two HIP events recorded on the
 * stream it is launched on (the events cost a few microseconds per launch).
 * Off by default. */
epic_status epic_ctx_set_timing(epic_ctx* ctx, int32_t enable);

/* Witness extraction (failure recovery, Sec. 4): how much of the search
 * state lives in LDS rather than in the witness workspace.  The back-trace
 * indexes up to max_proofs proofs in LDS, then moves its proof index to the
 * workspace for the rest of that sequence's search (0: the workspace's index
 * from the start); the byte search keeps a masked run's visited set in LDS
 * when it fits in max_vis_words 32-bit words, else in the workspace.  Where
 * they live changes only the speed, not which completions can be found.
 * 0 <= max_proofs <= 8192 and 0 <= max_vis_words <= 4096 (the defaults are
 * the maxima), else EPIC_ERR_ARG and the settings are unchanged.  Applies to
 * later epic_witness calls on the context. */
epic_status epic_ctx_set_witness_lds(epic_ctx* ctx, int32_t max_proofs, int32_t max_vis_words);

/* Diagnostics: synchronise `stream`, then read and clear, per kernel kind k
 * (0 lexing memo, 1 base walks of prefix sharing, 2 candidate walks of
 * validation, 3 selection (the walks it used: its own, and the helpers'
 * speculated walks whose results it took or drew an answer from),
 * 4 sequential fallback, 5 speculation bookkeeping (state clear, work
 * accounting), 6 speculated checks whose results the selection did not take
 * (no launches of their own, their time is the selection's)): ms[k]
 * the summed event durations of its timed launches, launches[k] their
 * number, work[k*6 .. k*6+5] the work counters of its walks (as
 * epic_ctx_work_counters).  Host arrays of 7, 7 and 42 elements. */
epic_status epic_ctx_kernel_stats(epic_ctx* ctx, hipStream_t stream, double* ms, int64_t* launches, int64_t* work);

/* Witness extraction for failure recovery (Sec. 4): when decoding stops
 * early, the output is completed from a witness of the current partial
 * sequence, which is completable because every committed update was checked.
 * For each sequence b of d_seqs (int32 [B*n], -1 = MASK), d_status[b]
 * (int32) is 1 when x_b is valid and a completion was found, 0 when x_b is
 * not valid, -1 when a token is out of range (EPIC_DEV_BAD_CANDIDATE), -2
 * when a buffer is too small (the witness workspace, bytes_per_seq or
 * max_gaps; EPIC_DEV_CAPACITY), -3 when no completion was found (not expected
 * for a valid x_b).  With status 1, d_gap_len[b*max_gaps + j] (int32) is the
 * number of bytes that fill the j-th maximal masked run of x_b, and
 * d_bytes[b*bytes_per_seq ..] holds the bytes of the runs in order: x_b with
 * every run replaced by its bytes lexes into a sentence of L(G).  A masked
 * run reads any byte string (the paper's over-approximation of masked
 * regions), so a filling is a byte string, not a number of tokens.
 * d_witness_ws: device memory of epic_witness_workspace_bytes(ctx, B) bytes,
 * 256-byte aligned, owned by the caller; d_workspace is the context's
 * workspace (its chart slots hold the walks).  B may not exceed the walk
 * slots of the context (min(max(max_cands, max_batch), 1024)):
 * EPIC_ERR_CAPACITY.  Asynchronous on stream. */
size_t epic_witness_workspace_bytes(const epic_ctx* ctx, int32_t B);
epic_status epic_witness(epic_ctx* ctx, const int32_t* d_seqs, int32_t B, int32_t n, uint8_t* d_bytes,
                         int32_t bytes_per_seq, int32_t* d_gap_len, int32_t max_gaps, int32_t* d_status,
                         void* d_witness_ws, size_t witness_ws_bytes, void* d_workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* Diagnostics: LDS streaming microbenchmark, the measurement behind the LDS
 * peak that walk kernels are compared with.  Launches `blocks` workgroups of
 * `threads` threads (a multiple of 64, at most 1024) on `stream`; each
 * workgroup fills 64 KiB of LDS, then every thread reads `iters` 16-byte
 * vectors from it at consecutive addresses (no bank conflicts), so the
 * launch reads blocks * threads * iters * 16 bytes of LDS.  d_sink: device
 * uint32 [8]; workgroup 0's thread 0 writes the shader-clock ticks (sink[2],
 * sink[3]: low, high word) and the constant-rate wall-clock ticks (sink[4],
 * sink[5]) it measured around its read loop; the caller times the launch
 * with events on the same stream.  Returns EPIC_ERR_ARG for sizes out of
 * range. */
epic_status epic_diag_lds_stream(int32_t blocks, int32_t threads, int32_t iters, uint32_t* d_sink,
                                 hipStream_t stream);

/* Shader-clock and wall-clock rates of the current device in kHz (as the
 * runtime reports them), for epic_diag_lds_stream's tick counts. */
epic_status epic_diag_clock_rates(int32_t* shader_khz, int32_t* wall_khz);

const char* epic_status_string(epic_status s);

#ifdef __cplusplus
}
#endif

#endif /* EPIC_H */
