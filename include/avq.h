/*
 * avq.h - C ABI of the MI355X (gfx950) AVQ-Attention forward pass.
 *
 * AVQ-Attention (Adaptive Vector-Quantized Attention) replaces keys by
 * codewords of a two-level codebook: M0 parents per head, each with Ch
 * children whose mean is the parent (Sec. 4.1, Eq. (parent_constraint)).
 * The forward pass is split into three calls, in this order:
 *
 *   avq_assign         keys -> nearest parent, then nearest child of that
 *                      parent (Sec. 4.2, Alg. 1)
 *   avq_aggregate      per-codeword key counts and value sums
 *                      (Eq. (aggregates), Alg. 1)
 *   avq_pack_aggregates  value sums and counts held by the caller, in the
 *                      operand layout of the attention kernel
 *   avq_attention_fwd  parent attention, per-query-tile importance, top-P
 *                      parent selection, child refinement with correcting
 *                      attention and normalisation (Sec. 4.3,
 *                      Eq. (vqflashattention), (importance),
 *                      (parent_recovery), (correcting_attention), Alg. 2)
 *   avq_attention_fwd_tiled  the same with the tiled-codeword importance of
 *                      App. B (Eq. (aproxdenom), (codewordimportance))
 *   avq_codebook_update  EMA codebook statistics and the constrained child
 *                      projection (App. A, Eq. (child_constraint_solve))
 *   avq_attention_fwd_ordered  attention with the queries in a given order
 *                      (the space-filling-curve reordering of Sec. 4)
 *   avq_gilbert_order  host helper: that order for a 2-D grid of tokens
 *
 * Conventions shared by every call:
 *   - Every array argument is a DEVICE pointer owned by the caller, contiguous,
 *     row-major and 16-byte aligned. Inputs are never written. Outputs are
 *     fully overwritten.
 *   - Tensors: Q, K, V, Y are [B][H][N][d]; the codebook is Cp [H][M0][d]
 *     (parents) and Cc [H][M0][Ch][d] (children of parent p in rows
 *     p*Ch .. p*Ch+Ch-1), shared across the batch (one codebook per head).
 *   - Codes: Mtot = M0*(1+Ch). Code p < M0 is parent p; code M0 + p*Ch + c is
 *     child c of parent p.
 *   - dtype selects the element type of Q, K, V, Cp, Cc and Y: AVQ_F32 (fp32)
 *     or AVQ_BF16 (bfloat16). Value sums are fp32, counts int32; the packed
 *     aggregates hold mean values in dtype.
 *   - Logits are exactly Q.C (the paper leaves the 1/sqrt(d) scale out of its
 *     formulas, Eq. (standardattention)); callers fold any scale into Q.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream). No call synchronises the device or allocates device memory:
 *     the device calls enqueue kernels only (no memset or copy), so after one
 *     call of an entry point on a device (it caches the device's attributes
 *     and kernel settings) its calls can be captured in a HIP graph.
 *   - Arguments are validated on the host before anything is launched; a
 *     non-OK status means nothing was enqueued (AVQ_ERR_DEVICE: a launch was
 *     rejected). avq_last_error() then returns a message for the calling
 *     thread. Inputs are not checked for NaN or infinity; the kernels are
 *     compiled without NaN semantics, so outputs for such inputs are
 *     unspecified (they need not be NaN).
 *   - Supported: d in {64, 128}; Ch in {0, 1, 2, 4, 8, 16}; 1 <= M0 <= 512;
 *     1 <= N <= 2^24, B >= 1, H >= 1 and B*H*N*d < 2^31. Other shapes return
 *     AVQ_ERR_UNSUPPORTED.
 *   - Ch = 0 is a flat codebook of M0 codewords (plain vector quantisation,
 *     Sec. 3.2): Cc may then be NULL, every code is a parent (Mtot = M0),
 *     and avq_attention_fwd needs P = 0, which is VQ attention (Sec. 3.2).
 */
#ifndef AVQ_H
#define AVQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AVQ_OK = 0,
  AVQ_ERR_INVALID_ARG = 1, /* null pointer, non-positive size, P outside [0, M0], ... */
  AVQ_ERR_UNSUPPORTED = 2, /* valid, but a shape/dtype this build has no kernel for */
  AVQ_ERR_DEVICE = 3       /* the HIP runtime rejected a launch */
} avq_status_t;

/* Element type of the dtype arguments. A plain 32-bit integer rather than an
 * enum type, so that any value a caller passes is well defined on arrival:
 * values other than these two are rejected with AVQ_ERR_INVALID_ARG. */
typedef int32_t avq_dtype_t;
enum { AVQ_F32 = 0, AVQ_BF16 = 1 };

/* Version of this ABI (major * 100 + minor). */
int avq_version(void);

/* Message for the last non-OK status returned to the calling thread
 * ("" if none). The pointer stays valid until the thread's next call. */
const char* avq_last_error(void);

/*
 * avq_assign - tree vector quantisation of the keys (Sec. 3.2 assignment with
 * squared Euclidean distance; Sec. 4.2 and Alg. 1 parent/child loops).
 *
 * For every key K[b][h][j]:
 *   parent_idx = p* = argmin_p ||K_j - Cp[h][p]||^2, lowest p on exact ties;
 *   c*            = argmin_c ||K_j - Cc[h][p*][c]||^2, lowest c on exact ties;
 *   code_idx      = M0 + p* * Ch + c* if that child distance is strictly below
 *                   the parent distance, else p* (always p* when Ch = 0).
 * Distances are evaluated in fp32 from the stored inputs.
 *
 *   K            [B][H][N][d]   dtype
 *   Cp           [H][M0][d]     dtype
 *   Cc           [H][M0][Ch][d] dtype (NULL allowed when Ch = 0)
 *   parent_idx   [B][H][N]      int32, out
 *   code_idx     [B][H][N]      int32, out
 */
avq_status_t avq_assign(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                        int32_t M0, int32_t Ch, const void* K, const void* Cp,
                        const void* Cc, int32_t* parent_idx, int32_t* code_idx,
                        void* stream);

/*
 * Bytes of the packed aggregates of one (batch, head) (see avq_aggregate) for
 * the given dtype and sizes. Returns -1 for an unknown dtype or sizes outside
 * 1 <= M0 <= 512, 0 <= Ch <= 16, 1 <= d <= 128.
 */
int64_t avq_packed_bytes(avq_dtype_t dtype, int32_t M0, int32_t Ch, int32_t d);

/*
 * avq_aggregate - per-codeword counts and value sums (Eq. (aggregates)).
 *
 * Parent rows p < M0 cover the whole parent cell (every key whose nearest
 * parent is p, whether or not it moved to a child: Alg. 1 adds to the parent
 * unconditionally); child rows M0 + p*Ch + c cover the keys that moved to
 * that child. The parent of a key is code_idx itself when code_idx < M0 and
 * (code_idx - M0) / Ch otherwise.
 *
 *   V         [B][H][N][d]      dtype
 *   code_idx  [B][H][N]         int32, values in [0, Mtot) (as avq_assign writes;
 *                               other values are ignored)
 *   Vbar      [B][H][Mtot][d]   fp32, out, nullable (the sums)
 *   counts    [B][H][Mtot]      int32, out
 *   packed    [B][H][E] bytes, out, nullable; E = avq_packed_bytes(): the
 *             aggregates in the operand layout avq_attention_fwd reads. Codes
 *             are grouped in octets of 8; the octets are, in order, the parents
 *             (parents 8o .. 8o+7, padded with empty octets to a multiple of 8
 *             octets), then for every parent p its ceil(Ch/8) child octets
 *             (children 8j .. 8j+7 of p), then one empty octet. The buffer is
 *               means [n_oct][d][8] in dtype: mean value Vbar/n of each code
 *                     of the octet (0 for n = 0 and for padding slots),
 *                     rounded from fp32;
 *               info  [n_oct][16] fp32: n of each code (slots 0..7) and ln n
 *                     (slots 8..15; -inf for n = 0 and padding);
 *             means first, info right after it.
 * At least one of Vbar and packed must be given.
 *
 * Every sum is accumulated in fp32 by the one half wave that owns the parent
 * family, keys in bucket order; counts are exact.
 */
avq_status_t avq_aggregate(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                           int32_t M0, int32_t Ch, const void* V, const int32_t* code_idx,
                           float* Vbar, int32_t* counts, void* packed, void* stream);

/*
 * avq_assign_aggregate - Alg. 1 as one precompute: the tree quantisation of
 * avq_assign and the counts and sums of avq_aggregate, with the child compare
 * and the value sums in one pass over each head's keys (Sec. 4.2: the
 * aggregates are formed in the same pass that assigns the keys).
 *
 * Outputs are those of avq_assign followed by avq_aggregate on its codes:
 * parent_idx and code_idx exactly (the same compare routine), counts exactly,
 * Vbar and packed within fp32 summation-order rounding. Two launches: the
 * parent assignment (it writes parent_idx, which the second launch reads),
 * then the child compare and aggregation per (batch, head, range of parent
 * families). Ch = 0 and Ch = 16 run avq_assign's two kernels and then
 * avq_aggregate's.
 *
 *   K, V         [B][H][N][d]   dtype
 *   Cp           [H][M0][d]     dtype
 *   Cc           [H][M0][Ch][d] dtype (NULL allowed when Ch = 0)
 *   parent_idx   [B][H][N]      int32, out
 *   code_idx     [B][H][N]      int32, out
 *   Vbar, counts, packed        as for avq_aggregate (Vbar or packed may be
 *                               NULL, not both)
 */
avq_status_t avq_assign_aggregate(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                  int32_t d, int32_t M0, int32_t Ch, const void* K,
                                  const void* V, const void* Cp, const void* Cc,
                                  int32_t* parent_idx, int32_t* code_idx, float* Vbar,
                                  int32_t* counts, void* packed, void* stream);

/*
 * avq_pack_aggregates - the aggregates in the form Alg. 2 takes them (its
 * input: the value sum Vbar and the count n of every code, Eq. (aggregates))
 * packed into the operand layout that avq_attention_fwd reads (the packed
 * buffer described under avq_aggregate). A caller that holds (Vbar, n) from
 * elsewhere reaches the attention kernel through this call.
 *
 * For every code x with n = max(counts[x], 0): mean = Vbar[x] * fl(1/n) in
 * fp32 (0 for n = 0), rounded once to dtype; info n (as a float) and
 * ln n = log2(n) ln 2 (-inf for n = 0); padding slots and the empty octet as
 * in avq_aggregate. This is the aggregation's own arithmetic: the Vbar and
 * counts that avq_aggregate writes pack into exactly its packed output.
 *
 *   Vbar     [B][H][Mtot][d]  fp32, rows as in avq_aggregate (parent rows the
 *                             whole cell, child rows the keys moved there)
 *   counts   [B][H][Mtot]     int32 (negative entries count as 0)
 *   packed   [B][H][E] bytes, out; E = avq_packed_bytes(dtype, M0, Ch, d)
 * Sizes as for avq_aggregate (N does not apply).
 */
avq_status_t avq_pack_aggregates(avq_dtype_t dtype, int32_t B, int32_t H, int32_t d,
                                 int32_t M0, int32_t Ch, const float* Vbar,
                                 const int32_t* counts, void* packed, void* stream);

/*
 * avq_attention_fwd - the fused refined-codebook attention (Alg. 2).
 *
 * Queries are taken in tiles of block_q consecutive tokens (the last tile may
 * be shorter). For each tile I and query i in I:
 *   parent pass  S_ip = Q_i . Cp_p; running max over non-empty parents
 *                (App. D); A_ip = exp(S_ip - m_i), zero for empty parents;
 *                Xbar_i = sum_p A_ip Vbar_p, Zbar_i = sum_p A_ip n_p
 *                (Eq. (vqflashattention));
 *   importance   w_p(I) = sum_{i in I} A_ip n_p / Zbar_i (Eq. (importance));
 *   top-P        the P parents of largest w (lowest index on ties);
 *   children     for every selected p and child c: T_ic = Q_i . Cc_pc; the
 *                running max is raised over non-empty children and Xbar, Zbar
 *                rescaled; the parent logit is recovered as the mean of all Ch
 *                child logits (Eq. (parent_recovery)); the correcting weight
 *                dA = exp(T_ic - m) - exp(Srec_ip - m), zero for empty children
 *                (Eq. (correcting_attention)), adds dA * Vbar_pc to Xbar and
 *                dA * n_pc to Zbar;
 *   output       Y_i = Xbar_i / Zbar_i.
 * P = 0 gives plain VQ attention over the parents (Sec. 3.2).
 *
 *   P            0 <= P <= M0; P = 0 when Ch = 0
 *   block_q      query tile size, 1 <= block_q <= 256 (semantic: importance
 *                and top-P are computed per tile of block_q tokens)
 *   Q            [B][H][N][d]    dtype
 *   Cp, Cc       as in avq_assign (Cc NULL allowed when Ch = 0)
 *   packed       the packed aggregates written by avq_aggregate or by
 *                avq_pack_aggregates (required)
 *   Y            [B][H][N][d]    dtype, out
 *   topp_idx     [B][H][T][P]    int32, out, nullable; T = ceil(N / block_q);
 *                the selected parents in the order importance descending,
 *                index ascending
 *   importance   [B][H][T][M0]   fp32, out, nullable; w_p(I) of every parent
 *
 * The kernel uses the log-count bias of App. D: a code's weight is
 * exp(S + ln n - m) applied to its mean value Vbar/n, which equals
 * exp(S - m) applied to Vbar; empty codes (n = 0) drop out without masks.
 *
 * Arithmetic: bf16 inputs use bf16 MFMA with fp32 accumulation (the weights
 * and the mean values are bf16 MFMA operands; softmax state, importance and
 * all sums stay fp32); fp32 inputs use fp32 MFMA throughout.
 */
avq_status_t avq_attention_fwd(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                               int32_t d, int32_t M0, int32_t Ch, int32_t P,
                               int32_t block_q, const void* Q, const void* Cp,
                               const void* Cc, const void* packed, void* Y,
                               int32_t* topp_idx, float* importance,
                               void* stream);

/* Parents per codeword tile of avq_attention_fwd_tiled. */
#define AVQ_IMPORTANCE_TILE 64

/*
 * avq_attention_fwd_tiled - avq_attention_fwd with the importance of App. B
 * (computing importance with tiled codewords), in one parent sweep.
 *
 * The parents are visited in tiles of AVQ_IMPORTANCE_TILE (parents
 * 64t .. 64t+63). After tile J the partial denominator of query i, the sum of
 * A_ip n_p over the parents of tiles up to J, is extrapolated to all keys
 * (Eq. (aproxdenom)): Ztilde_i(J) = N / N_seen(J) * partial, N_seen(J) being
 * the number of keys whose parent lies in those tiles; the importance of each
 * parent p of tile J is w_p(I) = sum_{i in I} A_ip n_p / Ztilde_i(J)
 * (Eq. (codewordimportance)). A tile whose parents hold no key adds nothing.
 * The last tile has N_seen = N, so with M0 <= AVQ_IMPORTANCE_TILE this is
 * Eq. (importance) and the call equals avq_attention_fwd. Top-P, the child
 * pass and the output are as in avq_attention_fwd, on this importance.
 *
 * Arguments, layouts, ownership, arithmetic and errors as avq_attention_fwd
 * (importance, when given, receives this w).
 */
avq_status_t avq_attention_fwd_tiled(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                     int32_t d, int32_t M0, int32_t Ch, int32_t P,
                                     int32_t block_q, const void* Q, const void* Cp,
                                     const void* Cc, const void* packed, void* Y,
                                     int32_t* topp_idx, float* importance, void* stream);

/*
 * avq_attention_fwd_ordered - avq_attention_fwd (tiled_importance = 0) or
 * avq_attention_fwd_tiled (tiled_importance = 1) with the queries taken in
 * the order query_order instead of token order: query tile t is the tokens
 * query_order[t*block_q .. t*block_q + block_q - 1]. The result equals
 * permuting the rows of Q by query_order, calling the unordered entry point
 * and writing each output row back to its token: Y[b][h][query_order[k]] is
 * the output of query position k. The reordering is the one the paper
 * applies before tiling (Sec. 4, along a space-filling curve; see
 * avq_gilbert_order), so that the tokens of a tile, which share one top-P
 * selection, are spatial neighbours. Keys, values and the aggregates are
 * order-free (Sec. 3.2) and are not reordered.
 *
 *   query_order  [N] int32, device, a permutation of 0 .. N-1 shared by every
 *                batch entry and head. An entry outside [0, N) makes that
 *                query position take no part (no output row is written for
 *                it); a repeated entry writes that token's row more than once,
 *                in an unspecified order, and leaves some token unwritten.
 *   topp_idx, importance  per tile of the ORDERED queries.
 * Other arguments, layouts, ownership and errors as avq_attention_fwd.
 */
avq_status_t avq_attention_fwd_ordered(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                       int32_t d, int32_t M0, int32_t Ch, int32_t P,
                                       int32_t block_q, const int32_t* query_order,
                                       int32_t tiled_importance, const void* Q, const void* Cp,
                                       const void* Cc, const void* packed, void* Y,
                                       int32_t* topp_idx, float* importance, void* stream);

/*
 * avq_gilbert_order - host helper: the cells of a width x height grid of
 * tokens (token y*width + x) in the order of a generalized Hilbert curve
 * (the Gilbert curve the paper reorders tokens along, Sec. 4,
 * Fig. per-tile adaptivity, App. spatial reordering ablation).
 *
 * The curve starts at cell (0, 0), visits every cell once, and each step
 * moves to a 4-neighbour, except for at most one diagonal step on some grids
 * with odd sides; on a 2^k x 2^k grid it is a Hilbert curve. Any run of
 * consecutive cells therefore covers a compact region, whatever the tile size.
 *
 *   width, height  grid sizes, >= 1, width*height <= 2^24
 *   order          [width*height] int32, HOST, out: order[k] = token of the
 *                  k-th cell (the query_order of avq_attention_fwd_ordered)
 *   rank           [width*height] int32, HOST, out, nullable: the inverse,
 *                  rank[order[k]] = k
 * Runs on the host only (no device call); copy order to the device once.
 */
avq_status_t avq_gilbert_order(int32_t width, int32_t height, int32_t* order, int32_t* rank);

/*
 * avq_codebook_update - one step of the codebook's exponential moving
 * averages under the parent-child constraint (App. A).
 *
 * The batch statistics are the aggregates of the KEYS (avq_aggregate called
 * with K in place of V, after avq_assign): sums[b][h][x] is the sum of the
 * keys with code x in batch entry b (a parent row covers its whole cell) and
 * counts[b][h][x] their number. For every head h (one codebook per head,
 * shared by the batch) and code x, summing over b in order:
 *   S_x <- lambda S_x + (1 - lambda) sum_b sums[b][h][x]
 *   N_x <- lambda N_x + (1 - lambda) sum_b counts[b][h][x]
 * Parents take the unconstrained mean C_p = S_p / N_p. The Ch children of p,
 * with means M_c = S_c / N_c, are projected onto the constraint that their
 * mean is C_p by the mass-weighted least-squares solution
 * (Eq. (child_constraint_solve)):
 *   delta = sum_c M_c - Ch C_p,  sigma = sum_c 1 / N_c,
 *   C_pc  = M_c - delta / (N_c sigma).
 *
 *   lambda   EMA decay, 0 < lambda <= 1 (else AVQ_ERR_INVALID_ARG)
 *   sums     [B][H][Mtot][d]  fp32 (the Vbar output of avq_aggregate on K)
 *   counts   [B][H][Mtot]     int32 (its counts)
 *   S        [H][Mtot][d]     fp32, in/out: the EMA key sums
 *   Nema     [H][Mtot]        fp32, in/out: the EMA counts; must be positive
 *                             on entry (then they stay positive); a
 *                             non-positive mass gives non-finite codewords
 *   Cp_out   [H][M0][d]       dtype, out: the new parents
 *   Cc_out   [H][M0][Ch][d]   dtype, out: the new children (NULL allowed
 *                             when Ch = 0)
 * Sizes as for the other calls (N does not apply). Arithmetic is fp32, one
 * thread per (family, dimension), batch entries summed in order; counts are
 * exact while the total count of a code stays below 2^24. The codewords are
 * rounded once to dtype.
 */
avq_status_t avq_codebook_update(avq_dtype_t dtype, int32_t B, int32_t H, int32_t d,
                                 int32_t M0, int32_t Ch, float lambda, const float* sums,
                                 const int32_t* counts, float* S, float* Nema, void* Cp_out,
                                 void* Cc_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* AVQ_H */
