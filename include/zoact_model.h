/*
 * zoact_model.h -- support operations of the forward-only ZO step (gfx950).
 *
 * The perturbed forward of Algorithm 2 runs the whole model, of which the adapted
 * linears (zoact.h) are the method's part; these calls are the rest of a decoder
 * forward for the Llama- and OPT-style models the paper fine-tunes (Section 5):
 * embeddings, normalisation, rotary position embedding and causal attention.  The
 * LM head is zoact_linear_fwd_pm with r = 0 and fp32 output; the SwiGLU / ReLU
 * activations and the residual additions are epilogues of zoact_linear_fwd_pm; the
 * loss is zoact_xent_pm.
 *
 * Conventions are those of zoact.h: device pointers, caller-owned buffers, host-side
 * validation before any enqueue (ZOACT_E_INVALID), stream-ordered, no allocation.
 * Activations are F32 or BF16 (dtype argument); norm weights and biases have the
 * activation type.  Rows of both perturbation halves are stacked: a [2][T][d] tensor
 * is 2T rows of d.
 */
#ifndef ZOACT_MODEL_H
#define ZOACT_MODEL_H

#include "zoact.h"

#ifdef __cplusplus
extern "C" {
#endif

/* out[h][t][:] = table[id][:] (+ pos[t % seq + pos_offset][:] if pos != NULL) for both
 * halves h = 0, 1 and t < n_tok, where id = tokens[t] when distinct_halves == 0 (the two
 * perturbations see the same input) and id = tokens[h * n_tok + t] when it is 1 (two
 * independent token sets, as in the unperturbed calibration forward of Algorithm 1).
 * tokens int32 [n_tok] or [2][n_tok] (ids must lie in [0, vocab); out-of-range ids are
 * clamped), table [vocab][d], pos [max_pos][d] or NULL (positions past max_pos are
 * clamped), out [2][n_tok][d]; the sum is formed in fp32 and rounded once. */
zoact_status zoact_embed(const int32_t* tokens, int64_t n_tok, int32_t distinct_halves, int64_t vocab,
                         const void* table, const void* pos, int64_t max_pos, int32_t pos_offset, int64_t seq,
                         int64_t d, int32_t dtype, void* out, zoact_stream stream);

/* y = x / sqrt(mean(x^2) + eps) * w per row (fp32 arithmetic, one rounding); x, y [rows][d]. */
zoact_status zoact_rmsnorm(const void* x, const void* w, int64_t rows, int64_t d, float eps, int32_t dtype, void* y,
                           zoact_stream stream);

/* y = (x - mean) / sqrt(var + eps) * w + b per row (biased variance); x, y [rows][d]. */
zoact_status zoact_layernorm(const void* x, const void* w, const void* b, int64_t rows, int64_t d, float eps,
                             int32_t dtype, void* y, zoact_stream stream);

/* Rotary position embedding (rotate-half) in place on columns [col0, col0 + n_heads *
 * head_dim) of rows of x (row stride ld elements): for each head and j < head_dim/2,
 * (lo, hi) = (x[j], x[j + head_dim/2]) becomes (lo c - hi s, hi c + lo s) with c, s from
 * the fp32 tables cos/sin [seq][head_dim/2] at position (row % seq).  fp32 arithmetic,
 * one rounding. */
zoact_status zoact_rope(void* x, int32_t dtype, int64_t rows, int64_t ld, int64_t col0, int32_t n_heads,
                        int32_t head_dim, int64_t seq, const float* cos_t, const float* sin_t, zoact_stream stream);

/* Causal attention over n_seq independent sequences of length seq (both halves and all
 * batch rows stacked): row t = b * seq + s.  q [rows][ldq] holds n_heads heads of
 * head_dim starting at column 0, k [rows][ldk] and v [rows][ldv] hold n_kv_heads heads
 * (head h reads kv head h / (n_heads / n_kv_heads)); out [rows][n_heads * head_dim].
 * Scores are fp32 (scaled by `scale`), softmax fp32; in bf16 the probabilities are rounded
 * to bf16 before multiplying V.  BF16 supports head_dim 64 or 128; F32 supports any
 * head_dim <= 128 with seq * head_dim <= 4096. */
zoact_status zoact_attention(const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                             int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                             float scale, int32_t dtype, void* out, zoact_stream stream);

/* zoact_rope on q (n_heads) and k (n_kv_heads) with the fp32 tables cos/sin
 * [seq][head_dim/2] (16-byte aligned), then zoact_attention: the same output bits as the
 * two calls.  Where the whole sequence is held in LDS (bf16, seq <= 256, four or more
 * query heads per key/value head, a grid of at least one workgroup per compute unit) the
 * rotation happens as q and k are read and the q and k buffers keep their values; else
 * they are rotated in place first.  So after the call q and k hold either the rotated or
 * the original values: callers treat them as consumed. */
zoact_status zoact_attention_rope(void* q, int64_t ldq, void* k, int64_t ldk, const void* v, int64_t ldv,
                                  int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                  float scale, int32_t dtype, const float* cos_t, const float* sin_t, void* out,
                                  zoact_stream stream);

/* Post-state of zoact_attention_rope for a configuration on the current device: 1 when
 * the call rotates q and k in place, 0 when it leaves them as they were.  Host only (no
 * GPU work); an invalid configuration (dtype other than F32/BF16, a count below 1, head
 * grouping that does not divide) gives -1. */
int32_t zoact_attention_rope_in_place(int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads,
                                      int32_t head_dim, int32_t dtype);

#ifdef __cplusplus
}
#endif
#endif /* ZOACT_MODEL_H */
