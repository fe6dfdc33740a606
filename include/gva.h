/*
 * gva.h -- C ABI of libgva.so, the MI355X (gfx950) decode step of Grouped
 * Value Attention with decoupled RoPE.
 *
 * One decode step (Algorithm 1 of the paper) is four calls:
 *
 *   gva_append_kv         write the new value rows and the rotated shared
 *                         positional key into the caches (Algorithm 1, the
 *                         append steps; eq. krope)
 *   gva_absorb_query      q~_h = q^nope_h M_h^T and q^rope_h R_p^T
 *                         (eq. absorb, Section 3.2; the query-rotation step)
 *   gva_decode_attention  per split of the cached rows: scores
 *                         q~ . V_g(h)[t] + q^rope . k^rope[t], scaled softmax
 *                         and the weighted value sum, never forming a
 *                         content key (Section 3.3; the scoring and output
 *                         steps of Algorithm 1)
 *   gva_combine           log-sum-exp merge of the split partials
 *
 * Paged caches (a block table over page pools) have their own append and
 * attention calls, gva_paged_append_kv and gva_paged_decode_attention.
 *
 * The matched grouped-query baseline the paper measures GVA against
 * (explicit key stream per group) has its own attention call,
 * gva_gqa_decode_attention, sharing the layout, splits and gva_combine.
 * GVA with ordinary RoPE (keys reconstructed and rotated per position, the
 * variant that cannot absorb M_h) has gva_rope_decode_attention, as a
 * contrast workload.  A prompt is attended causally in one pass with
 * gva_prefill_absorb + gva_prefill_attention (gva_gqa_prefill_attention
 * for the matched GQA baseline).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every tensor argument is a DEVICE pointer to a dense, row-major array;
 *   only `dims` is a host pointer.  The caller owns all memory.  The library
 *   never allocates, frees or synchronises; each call enqueues its kernels
 *   on `stream` (a hipStream_t; NULL is the null stream) and returns.
 * - Storage dtype (`dims->dtype`) applies to q, M, the caches and the new
 *   rows: GVA_DTYPE_BF16 (bfloat16) or GVA_DTYPE_F32.  Absorbed queries,
 *   partials and outputs are always fp32.
 * - Layouts (B batch, H query heads, G value groups, T = dims->t_max):
 *     q        [B][H][d_c + d_r]   content slice first, then the positional
 *                                  slice, unrotated
 *     M        [H][d_v][d_c]       M_h maps a d_v-wide value to a d_c-wide
 *                                  content key (K_h = V_g(h) M_h, eq. kvm)
 *     v_cache  B*G streams of T rows x d_v   grouped value cache
 *     kr_cache B streams of T rows x d_r     shared positional key cache,
 *                                  stored already rotated
 *   Both caches use the tiled layout below (their total sizes equal the
 *   row-major [B][G][T][d_v] and [B][T][d_r] arrays).  They are written by
 *   gva_append_kv; a caller that fills them itself must follow the layout.
 *     lens     [B] int32           cached rows per sequence; the query sits
 *                                  at position lens[b]-1 (positions 0-based)
 * - Tiled cache layout.  Stream (b, g) of v_cache starts at element
 *   (b*G + g)*T*d_v, stream b of kr_cache at b*T*d_r.  With D the row width
 *   of the stream, E the element size and P = 16/E elements per 16-byte
 *   piece, element (t, i) of a stream sits at element offset
 *       (t/16)*16*D + ((i/P)*16 + t%16)*P + i%P
 *   i.e. tiles of 16 rows, inside a tile the 16-byte pieces of the rows
 *   ordered piece-major.  This lets one wave-wide 16-byte load fetch 1 KB of
 *   contiguous memory into matrix-core operand order.  It requires T % 16 ==
 *   0 and d_v, d_r multiples of P (8 for bf16, 4 for fp32).
 * - Head h reads value group g(h) = h / (H/G).
 * - RoPE rotates interleaved pairs (2i, 2i+1) by the angle
 *   p * rope_base^(-2i/d_r), formed in fp64, as the row-vector product
 *   x R_p^T: (x0 cos a - x1 sin a, x0 sin a + x1 cos a).
 * - Score scale: dims->scale, or 1/sqrt(d_c + d_r) when it is 0 (d_qk =
 *   d_n + d_r, Section 3.3).
 * - Device-resident indices are clamped, never trusted: lens[b] is read as
 *   min(max(lens[b], 0), T); append rows whose seq/pos fall outside
 *   [0,B) x [0,T) are skipped.
 * - Errors: every call returns a gva_status.  All arguments are validated
 *   on the host before anything is enqueued; a failed validation enqueues
 *   nothing.  GVA_ERR_HIP reports a launch failure from the HIP runtime.
 * - Calls are asynchronous; outputs must not alias inputs.  Results are
 *   bitwise deterministic for a fixed num_splits.
 */
#ifndef GVA_H_
#define GVA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gva_status {
  GVA_OK = 0,
  GVA_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad dims or split count */
  GVA_ERR_UNSUPPORTED = -2, /* valid shape the library has no kernel for */
  GVA_ERR_HIP = -3,         /* the HIP runtime reported an error */
  GVA_ERR_SCRATCH = -4      /* gva_decode_step_static: more than GVA_STATIC_SCRATCH_BYTES needed */
} gva_status;

typedef enum gva_dtype { GVA_DTYPE_F32 = 0, GVA_DTYPE_BF16 = 1 } gva_dtype;

/* Problem shape; passed by host pointer to every call. */
typedef struct gva_dims {
  int32_t batch;      /* B >= 1 */
  int32_t n_heads;    /* H >= 1, a multiple of n_groups */
  int32_t n_groups;   /* G >= 1 */
  int32_t d_v;        /* value width (the paper's d_h) */
  int32_t d_c;        /* content query/key width (the paper's d_n) */
  int32_t d_r;        /* shared positional width, even, >= 0 */
  int32_t t_max;      /* cache capacity per sequence, >= 1 */
  int32_t dtype;      /* gva_dtype */
  double rope_base;   /* RoPE base (10000 in the paper's setting), > 0 */
  double scale;       /* score scale; 0 selects 1/sqrt(d_c + d_r) */
} gva_dims;

/*
 * Paged caches (for ragged serving: a sequence's rows live in fixed-size
 * pages drawn from shared pools, found through a block table).
 *   v_pool  [n_pages][G][page_rows][d_v]   each (page, g) block in the
 *                                           tiled layout of a stream
 *   kr_pool [n_pages][page_rows][d_r]      each page block tiled likewise
 *   block_table [B][max_pages] int32       row t of sequence b is row
 *           t % page_rows of page block_table[b][t / page_rows]
 * page_rows is a positive multiple of 32; dims->t_max must equal
 * max_pages * page_rows (the capacity of a sequence); max_pages <=
 * GVA_MAX_PAGES.  Entries a call needs (the pages of rows below lens[b], or
 * of an appended position) must name pages in [0, n_pages): the attention
 * kernel clamps other ids into the pool (it reads some page, never outside
 * the pool) and the append skips rows whose page is out of range.  bf16
 * storage only.
 */
typedef struct {
  int32_t page_rows;
  int32_t max_pages;
  int32_t n_pages;
} gva_paging;

/* Largest max_pages accepted by the paged calls. */
#define GVA_MAX_PAGES 4096

/* Largest num_splits accepted by gva_decode_attention / gva_combine. */
#define GVA_MAX_SPLITS 256

/*
 * gva_append_kv -- Algorithm 1, the cache-append steps, and eq. krope.
 * For each r < n_rows, with b = seq[r], p = pos[r]:
 *   v_cache[b][g][p][:] = v_new[r][g][:]              for every g < G
 *   kr_cache[b][p][:]   = RoPE(kr_new[r][:], p)       rotated in fp64,
 *                                                     rounded once (RNE)
 * v_new [n_rows][G][d_v] and kr_new [n_rows][d_r] are device arrays in the
 * storage dtype; kr_new is the unrotated x W_r.  seq/pos are device int32
 * [n_rows].  Rows with b or p out of range are skipped.  Writing the same
 * (b, p) twice with the same data is idempotent; two rows naming the same
 * (b, p) in one call race.  n_rows == 0 is a no-op.
 * Pointers: v_cache, v_new, kr_cache 16-byte aligned; kr_new 4-byte
 * aligned (the last two only when d_r > 0).  Shapes outside the tiled
 * layout's requirements: GVA_ERR_UNSUPPORTED.
 */
int gva_append_kv(const gva_dims* dims, void* v_cache, void* kr_cache,
                  const void* v_new, const void* kr_new,
                  const int32_t* seq, const int32_t* pos, int32_t n_rows,
                  void* stream);

/*
 * gva_absorb_query -- eq. absorb (Section 3.2) and the query-rotation step
 * of Algorithm 1, for every (b, h):
 *   q_abs[b][h][i] = sum_k q[b][h][k] * M[h][i][k]        (q~ = q^nope M_h^T)
 *   q_rot[b][h][:] = RoPE(q[b][h][d_c : d_c+d_r], lens[b]-1)
 * Outputs are fp32 and unscaled.  q_rot may be NULL when d_r == 0.
 * bf16 needs d_v % 16 == 0, d_c % 32 == 0, d_r % 8 == 0 (matrix cores);
 * fp32 takes any shape.  q, m, q_abs 16-byte aligned.
 */
int gva_absorb_query(const gva_dims* dims, const void* q, const void* m,
                     const int32_t* lens, float* q_abs, float* q_rot, void* stream);

/*
 * gva_decode_attention -- the attention steps of Algorithm 1 over split s
 * of every sequence, for every (b, h, s):
 *   rows    P = [s*c_b, min(L_b, (s+1)*c_b)),  L_b = lens[b] (clamped to
 *           [0, T]),  S = num_splits,  c_b = 32 * ceil(ceil(L_b / n_b) / 32):
 *           the first n_b splits share the rows evenly and the rest are
 *           empty, with n_b = S when split_rows == 0 (even splits), else
 *           n_b = ceil(L_b / split_rows) clamped to [1, S] (bounded chunks:
 *           no split of more than split_rows rows unless S such splits
 *           cannot cover L_b, for batches of unequal lengths)
 *   score   x_t = scale * ( q~_h . v_cache[b][g(h)][t] + q^rope_h . kr_cache[b][t] )
 *   o_part[b][h][s][:] = sum_{t in P} softmax(x)_t v_cache[b][g(h)][t][:]
 *   lse_part[b][h][s]  = log sum_{t in P} exp(x_t)       (natural log)
 * An empty P writes lse_part = -inf; its o_part is written (zeros) only for
 * s = 0 and is otherwise left untouched (gva_combine never reads it).  With
 * S == 1 the partials are the final (o, lse).  split_rows must be a
 * non-negative multiple of 32.
 * The query comes either raw -- q and m non-NULL, q_abs and q_rot NULL: the
 * kernel absorbs and rotates it itself ahead of the attention loop (the
 * fused path) -- or pre-absorbed by gva_absorb_query: q/m NULL, q_abs
 * [B][H][d_v] fp32 and (if d_r > 0) q_rot [B][H][d_r] fp32 non-NULL.
 * In the fused path every workgroup absorbs its group's heads itself: it
 * suits launches of at most one workgroup per CU (B * G * num_splits) and
 * few splits; otherwise one gva_absorb_query call and the pre-absorbed
 * path cost less than every workgroup absorbing the same heads again.
 * The current token, appended and attended in one launch (optional):
 * v_new [B][G][d_v] and kr_new [B][d_r] (unrotated, storage dtype, as for
 * gva_append_kv) are the rows of position lens[b]-1 of every sequence with
 * lens[b] >= 1.  The call then stores them into the caches at that
 * position exactly as gva_append_kv does (same rotation and rounding) and
 * attends over them without reading them back, so the result equals
 * gva_append_kv followed by this call without the new rows.  Pass both
 * NULL when the caches already hold row lens[b]-1; kr_new may be NULL when
 * d_r == 0.  v_new 16-byte aligned, kr_new 4-byte aligned.
 * o_part [B][H][S][d_v] fp32, lse_part [B][H][S] fp32.
 * Supported for bf16: d_v in {64, 128}, d_c a multiple of 32 (<= 512),
 * d_r a multiple of 8 (<= 64), H/G in {1, 2, 4, 8}; for fp32: d_v <= 256,
 * d_c <= 512, d_r <= 64, H/G <= 8.  Other valid shapes: GVA_ERR_UNSUPPORTED.
 * Every shape must also satisfy the tiled cache layout (T % 16 == 0).
 * Pointers: 16-byte aligned.
 */
int gva_decode_attention(const gva_dims* dims, const void* q, const void* m,
                         const float* q_abs, const float* q_rot,
                         void* v_cache, void* kr_cache,
                         const int32_t* lens, const void* v_new, const void* kr_new,
                         int32_t num_splits, int32_t split_rows, float* o_part, float* lse_part,
                         void* stream);

/*
 * gva_paged_append_kv -- gva_append_kv on paged caches: row pos[r] of
 * sequence seq[r] is written to row pos % page_rows of page
 * block_table[seq][pos / page_rows] of both pools, with the same rotation
 * and rounding.  Pools 16-byte aligned, block_table 4-byte aligned.
 */
int gva_paged_append_kv(const gva_dims* dims, const gva_paging* paging, void* v_pool, void* kr_pool,
                        const int32_t* block_table, const void* v_new, const void* kr_new,
                        const int32_t* seq, const int32_t* pos, int32_t n_rows, void* stream);

/*
 * gva_paged_decode_attention -- gva_decode_attention on paged caches: the
 * same scores, softmax, splits, partials and current-row append (into the
 * current row's page), every cache row read through the block table.
 * A split's page ids are read once into LDS; each 32-row tile lies in one
 * page.  Arguments as for gva_decode_attention, plus the paging and
 * block_table (device int32 [B][max_pages]).
 */
int gva_paged_decode_attention(const gva_dims* dims, const gva_paging* paging, const void* q,
                               const void* m, const float* q_abs, const float* q_rot, void* v_pool,
                               void* kr_pool, const int32_t* block_table, const int32_t* lens,
                               const void* v_new, const void* kr_new, int32_t num_splits,
                               int32_t split_rows, float* o_part, float* lse_part, void* stream);

/*
 * gva_gqa_decode_attention -- the matched grouped-query attention baseline
 * that GVA is measured against (Section 2, GQA; Section 3.4 compares the
 * caches): one explicit key stream per group, stored already rotated as a
 * standard GQA cache is, and no positional term.  For every (b, h, s):
 *   rows    P as in gva_decode_attention (same split rule and split_rows)
 *   score   x_t = scale * q[b][h][0 : d_v] . k_cache[b][g(h)][t]
 *   o_part[b][h][s][:] = sum_{t in P} softmax(x)_t v_cache[b][g(h)][t][:]
 *   lse_part[b][h][s]  = log sum_{t in P} exp(x_t)
 * with scale = dims->scale, or 1/sqrt(d_v) when it is 0.  The key width is
 * d_v; d_c, d_r and rope_base are not used.  Empty P and S == 1 behave as in
 * gva_decode_attention; gva_combine merges the partials.
 * q [B][H][q_stride] in the storage dtype (only the first d_v entries of a
 * row are read); k_cache and v_cache: B*G streams of T rows x d_v in the
 * tiled layout.  Read only: the caches are not modified.
 * Supported: bf16, d_v in {64, 128}, H/G in {1, 2, 4, 8}, q_stride a
 * multiple of 8, T % 16 == 0; other valid shapes: GVA_ERR_UNSUPPORTED.
 * q_stride < d_v: GVA_ERR_INVALID_ARG.  Pointers: 16-byte aligned.
 */
int gva_gqa_decode_attention(const gva_dims* dims, const void* q, int32_t q_stride,
                             const void* k_cache, const void* v_cache, const int32_t* lens,
                             int32_t num_splits, int32_t split_rows, float* o_part, float* lse_part,
                             void* stream);

/*
 * gva_rope_decode_attention -- the contrast workload: GVA with ordinary
 * RoPE instead of decoupled RoPE (Section 3.2, the variant whose key map
 * cannot be absorbed at decode).  Content keys are reconstructed per
 * position and rotated over their whole width d_c at their own position;
 * there is no shared positional key.  For every (b, h, s), with L the
 * clamped length and P = L - 1 the query's position:
 *   rows    as in gva_decode_attention (same split rule and split_rows)
 *   key     k_t = RoPE(v_cache[b][g(h)][t] M_h, t)       (width d_c)
 *   score   x_t = scale * RoPE(q[b][h], P) . k_t
 *   o_part[b][h][s][:] = sum_{t in P} softmax(x)_t v_cache[b][g(h)][t][:]
 *   lse_part[b][h][s]  = log sum_{t in P} exp(x_t)
 * RoPE rotates interleaved pairs (2i, 2i+1) by t * rope_base^(-2i/d_c);
 * scale = dims->scale, or 1/sqrt(d_c) when it is 0.  The kernel evaluates
 * the scores through the equivalent per-pair form
 *   sum_i (v_t . W_h[:, 2i]) cos(theta_i (t-P)) + (v_t . W_h[:, 2i+1]) sin(theta_i (t-P))
 * with W_h built from q and M_h once per workgroup and rounded to bf16, so
 * every position still costs d_v * d_c multiply-adds per head; this
 * rounding and the fp32 cos/sin make it less exact than the absorbed path.
 * Empty splits and S == 1 behave as in gva_decode_attention; gva_combine
 * merges the partials.  The current token's value row must already be in
 * the cache (gva_append_kv with d_r = 0); the caches are only read.
 * dims->d_r must be 0 and d_c even: else GVA_ERR_INVALID_ARG.
 * q [B][H][d_c] and M [H][d_v][d_c] in bf16; v_cache B*G streams of
 * T rows x d_v in the tiled layout.
 * Supported: bf16, d_v and d_c in {64, 128}, H/G in {1, 2, 4, 8} with
 * H/G * d_v * d_c * 2 bytes <= 128 KiB; other valid shapes:
 * GVA_ERR_UNSUPPORTED.  Pointers: 16-byte aligned (lens 4).
 */
int gva_rope_decode_attention(const gva_dims* dims, const void* q, const void* m, const void* v_cache,
                              const int32_t* lens, int32_t num_splits, int32_t split_rows,
                              float* o_part, float* lse_part, void* stream);

/*
 * Prefill: causal attention for a prompt of n_new tokens per sequence, after
 * any cached prefix (Algorithm 1's loop for every prompt position at once;
 * Section 3.3's scores; training uses the same split with standard causal
 * attention).  The prompt's rows are appended first (gva_append_kv with
 * n_new rows per sequence), so each sequence's n_new query rows are its
 * last n_new cached rows: query i of sequence b sits at position
 * p = L_b - n_new + i (L_b = lens[b], clamped to [0, T]) and sees rows 0..p.
 * Rows with p < 0 (L_b < n_new) get o = 0, lse = -inf.
 *
 * gva_prefill_absorb -- gva_absorb_query for every query row: q is
 * [B][n_new][H][d_c+d_r] in the storage dtype; q_abs [B][n_new][H][d_v]
 * and q_rot [B][n_new][H][d_r] fp32, the positional slice rotated at the
 * row's own position.  B * n_new <= 2^20.  1 <= n_new <= T, else
 * GVA_ERR_INVALID_ARG.
 */
int gva_prefill_absorb(const gva_dims* dims, int32_t n_new, const void* q, const void* m,
                       const int32_t* lens, float* q_abs, float* q_rot, void* stream);

/*
 * gva_prefill_attention -- for every (b, i, h) with p >= 0:
 *   score   x_t = scale * ( q_abs[b][i][h] . V[b][g(h)][t] + q_rot[b][i][h] . kr[b][t] ),  t <= p
 *   o[b][i][h][:] = sum_{t <= p} softmax(x)_t V[b][g(h)][t][:]
 *   lse[b][i][h]  = log sum_{t <= p} exp(x_t)
 * with scale as in gva_decode_attention.  A dense contraction, unlike the
 * bandwidth-bound decode step (which keeps query and weights as bf16
 * high+low pairs): the queries enter the matrix cores as bf16, the softmax
 * weights and the value rows as fp16 (exact for bf16 values of magnitude
 * 2^-14 .. 65504; value entries must stay below 65504 in magnitude).
 * o [B][n_new][H][d_v] fp32, lse [B][n_new][H] fp32; the caches are read
 * only.  Supported: bf16, d_v in {64, 128}, d_r a multiple of 8 (<= 64),
 * H/G in {1, 2, 4, 8}, T % 16 == 0; other valid shapes:
 * GVA_ERR_UNSUPPORTED.  Pointers 16-byte aligned (lens, lse 4).
 */
int gva_prefill_attention(const gva_dims* dims, int32_t n_new, const float* q_abs, const float* q_rot,
                          const void* v_cache, const void* kr_cache, const int32_t* lens, float* o,
                          float* lse, void* stream);

/*
 * gva_gqa_prefill_attention -- the matched grouped-query prefill the paper
 * compares GVA against: the same causal rows, scores q[b][i][h] . k_cache
 * [b][g(h)][t] over an explicit key stream of width d_v (no positional
 * term; scale = dims->scale or 1/sqrt(d_v)).  q [B][n_new][H][d_v] fp32;
 * k_cache like v_cache.  Shapes and outputs as for gva_prefill_attention;
 * d_c, d_r and rope_base are not used.
 */
int gva_gqa_prefill_attention(const gva_dims* dims, int32_t n_new, const float* q, const void* k_cache,
                              const void* v_cache, const int32_t* lens, float* o, float* lse,
                              void* stream);

/*
 * gva_combine -- log-sum-exp merge of split partials, for every (b, h):
 *   LSE = log sum_s exp(lse_part[b][h][s]);
 *   o[b][h][:] = sum_s exp(lse_part[b][h][s] - LSE) * o_part[b][h][s][:]
 * Partials with lse = -inf do not contribute, whatever their o_part holds
 * (the first eight of a row are requested together with the LSEs, before
 * it is known which are empty; later ones only when non-empty); if all are
 * empty, o = 0 and LSE = -inf.
 * lse may be NULL.  o [B][H][d_v] fp32, lse [B][H] fp32; d_v <= 256.
 */
int gva_combine(const gva_dims* dims, const float* o_part, const float* lse_part,
                int32_t num_splits, float* o, float* lse, void* stream);

/*
 * gva_decode_workspace_size, gva_decode_step -- one whole decode step of
 * Algorithm 1 in one call: the current token's rows appended (optional, as
 * in gva_decode_attention), the query absorbed and rotated (eq. absorb,
 * Section 3.2), the attention over every cached row in num_splits splits
 * (Section 3.3) and the log-sum-exp merge of the splits, for every (b, h):
 *   o[b][h][:] = sum_{t < L_b} softmax(x)_t v_cache[b][g(h)][t][:]
 *   lse[b][h]  = log sum_{t < L_b} exp(x_t)
 * with x_t as in gva_decode_attention (L_b = 0: o = 0, lse = -inf).  The
 * result equals, bit for bit, the calls gva_prefer_fused chooses for the
 * same plan on the current device: gva_decode_attention with the raw query,
 * or gva_absorb_query and then gva_decode_attention with its output; then
 * gva_combine when num_splits > 1.
 * The intermediate buffers -- the absorbed queries of the separate path and
 * the split partials -- live in `workspace`, a caller-owned device buffer of
 * at least the bytes gva_decode_workspace_size reports for the same dims,
 * num_splits and split_rows on the current device, 256-byte aligned (0
 * bytes for one split with the absorption fused: workspace may then be
 * NULL).  Its contents are scratch: nothing needs clearing before a call and
 * nothing of it is used after one.  q, m, the caches, lens, v_new, kr_new,
 * num_splits and split_rows as for gva_decode_attention (the raw query is
 * required); o [B][H][d_v] fp32 and lse [B][H] fp32, both required.  Every
 * launch is validated before the first is enqueued; a workspace that is
 * missing, short or misaligned: GVA_ERR_INVALID_ARG.
 */
int gva_decode_workspace_size(const gva_dims* dims, int32_t num_splits, int32_t split_rows, size_t* bytes);
int gva_decode_step(const gva_dims* dims, const void* q, const void* m, void* v_cache, void* kr_cache,
                    const int32_t* lens, const void* v_new, const void* kr_new, int32_t num_splits,
                    int32_t split_rows, void* workspace, size_t workspace_bytes, float* o, float* lse,
                    void* stream);

/*
 * gva_decode_step_static -- gva_decode_step for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same launches, bit for bit
 * the same results, with the workspace taken from the library's static
 * scratch buffer instead of an argument.  The buffer is a file-scope device
 * array of GVA_STATIC_SCRATCH_BYTES, one on every GPU the library runs on,
 * held until the process ends; its address is looked up on the first call
 * on each device.  The call allocates, frees and clears nothing.  A plan
 * whose workspace (gva_decode_workspace_size) exceeds the buffer returns
 * GVA_ERR_SCRATCH and enqueues nothing.  Every call on a GPU shares that
 * GPU's buffer: calls that may run at the same time on one GPU (different
 * streams, or host threads) race and must be ordered by the caller; calls
 * in one stream are ordered already.  Arguments as for gva_decode_step.
 */
#define GVA_STATIC_SCRATCH_BYTES (16u << 20)
int gva_decode_step_static(const gva_dims* dims, const void* q, const void* m, void* v_cache, void* kr_cache,
                           const int32_t* lens, const void* v_new, const void* kr_new, int32_t num_splits,
                           int32_t split_rows, float* o, float* lse, void* stream);

/*
 * gva_pick_splits -- host heuristic: the split plan for a batch whose
 * longest sequence has max_len rows and whose lengths sum to total_len
 * (0 = unknown: every sequence taken as max_len), on a device with n_cu
 * compute units (0 = ask the current device).  Returns num_splits in
 * [1, GVA_MAX_SPLITS]; when split_rows is non-NULL it receives the
 * split_rows to pass with it (0 = even splits; bounded chunks are chosen for
 * widely spread lengths over more (sequence, group) streams than a quarter
 * of the compute units).  Even splits: one while the longest stream holds
 * less than 192 KiB of value rows, else about one workgroup per compute
 * unit, none under 32 KiB, at most 16.  With split_rows NULL the plan uses
 * even splits only.  Pure host code; enqueues nothing.
 */
int gva_pick_splits(const gva_dims* dims, int32_t max_len, int64_t total_len, int32_t n_cu,
                    int32_t* split_rows);

/*
 * gva_prefer_fused -- host heuristic: 1 if a gva_decode_attention launch of
 * num_splits splits (split_rows as for that call) should take the raw query
 * and absorb it in the attention kernel (the fused path), 0 if one
 * gva_absorb_query call ahead of it costs less.  The fused path pays for an
 * absorption in every workgroup (H/G maps of d_v x d_c, read from the
 * L2): it wins while all the launch's workgroups (B * splits rounded up to
 * 8, times G) are resident at once, two per CU on a device with n_cu
 * compute units (0 = ask the current device), or, with bounded chunks,
 * while a chunk's split_rows value rows are at least as many as the map
 * rows a workgroup reads (split_rows >= (H/G) d_c).  Returns 0 for
 * invalid dims.  Pure host code; enqueues nothing.
 */
int gva_prefer_fused(const gva_dims* dims, int32_t num_splits, int32_t split_rows, int32_t n_cu);

/* Human-readable name of a gva_status value (static storage). */
const char* gva_status_string(int status);

/* ABI version of this header: major * 10000 + minor * 100 + patch. */
int gva_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GVA_H_ */
