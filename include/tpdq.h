/*
 * tpdq.h - C ABI of libtpdq: TP-aware dequantization (arXiv 2402.04925) for
 * AMD Instinct MI355X (gfx950).
 *
 * The library computes the hot path of the paper's method on one GPU:
 *   - the offline reorder of an act-order GPTQ layer pair (Alg. 1, and the
 *     TP-aware fold of section 2.2 / Alg. 3's inputs W1[P1, P2] and W2[P2]);
 *   - the W4A16 dequantize-and-multiply, both with per-row metadata fetched
 *     through an unordered g_idx (Eq. 3, the load of Fig. 1) and with sorted
 *     rows whose group of row k is floor(k / G) (Eq. 1, the load of Fig. 2);
 *   - one rank's share of the TP-aware MLP, Alg. 3 without its AllReduce:
 *     Y1 = X[:, P1] @ W1_local, Y2 = Y1 @ W2_local.
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is DEVICE memory owned by the caller. The library
 *     never allocates device memory and never frees what it is given.
 *   - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL is the
 *     legacy default stream). Unless stated otherwise a call returns right
 *     after validation and launch; the results are ready when the stream is.
 *   - Matrices are row-major; every leading dimension `ld_*` is in elements
 *     of the array it describes.
 *   - Arguments are validated on the host before anything is enqueued: a
 *     non-OK status means no work was enqueued (except where stated for
 *     tpdq_reorder). tpdq_last_error() then gives a one-line reason.
 *   - Faults inside a kernel surface at the caller's next synchronisation.
 *   - Outputs must not alias inputs.
 *
 * Storage format of a quantized layer (the paper fixes none; this is the
 * GPTQ layout: group quantization of a K x N weight, section 1.1):
 *   qweight int32 [K/8][ld_q]   nibble j (bits 4j..4j+3) of word [r][n] is
 *                               the unsigned 4-bit code q of row 8r+j, col n
 *   scales  fp16 or bf16 [num_groups][ld_s]  one scale s per (group, column)
 *   qzeros  int32 [num_groups][ld_z]     nibble j of word [g][c] is the
 *                               4-bit zero code z of group g, column 8c+j
 *   g_idx   int32 [K]           group of row k
 *   dequantized weight: W[k][n] = s[g][n] * (q[k][n] - z[g][n]), g = g_idx[k],
 *   with z the stored zero code plus the layer's zero_offset
 * Groups: with a group size G > 0, Eq. 3 gives every group G rows except a
 * partial last group when G does not divide K (ceil(K/G) groups); a sorted
 * ("ordered") layer then has g_idx[k] == floor(k / G) (Eq. 1) and the ordered
 * kernels never read g_idx. G == 0 marks groups of unequal sizes given by
 * g_idx alone (a checkpoint's own grouping); a sorted layer of that kind is
 * read through its sorted (non-decreasing) g_idx.
 */
#ifndef TPDQ_H
#define TPDQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TPDQ_OK = 0,
  TPDQ_ERR_NULL = 1,        /* a required pointer is NULL                              */
  TPDQ_ERR_SHAPE = 2,       /* K%8, N%8, G%8, too few groups, K2 != N1, M < 1, ld too small */
  TPDQ_ERR_ALIGN = 3,       /* a pointer or leading dimension breaks the vector alignment */
  TPDQ_ERR_GIDX = 4,        /* g_idx out of range, or groups other than Eq. 3's (G > 0)  */
  TPDQ_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than tpdq_workspace_bytes()    */
  TPDQ_ERR_UNSUPPORTED = 6, /* valid request this build does not implement, e.g. a tensor of
                             2 GiB or more (the kernels address each tensor with 32-bit
                             byte offsets)                                             */
  TPDQ_ERR_HIP = 7          /* a HIP runtime call or a kernel launch failed             */
} tpdq_status;

/* Element type of X, the scales and the outputs (one type per call; the
 * paper's experiments use fp16, bf16 is the second type of the same
 * method). Both accumulate in fp32 and round the output to nearest even.
 * fp16: the ordered kernels subtract the zero exactly per element; the
 * act-order and prefill-sized kernels round each dequantized weight to fp16.
 * bf16: the ordered decode kernels keep q - z exact (the zero is applied per
 * group against the group's sum of X, so a product that is exactly 0 comes
 * out at fp32 rounding level, not 0); the act-order and prefill-sized
 * kernels round each dequantized weight to bf16. */
typedef enum { TPDQ_FP16 = 0, TPDQ_BF16 = 1 } tpdq_dtype;

/* Storage order of qweight.
 * TPDQ_LAYOUT_GPTQ: int32 [K/8][ld_q], word [r][n] = rows 8r..8r+7 of column n.
 * TPDQ_LAYOUT_TILED: the same words regrouped so that one wavefront of the
 *   decode GEMM reads 1 KB contiguous per load: int32 [ceil(N/16)][ld_q] with
 *   ld_q >= ceil(K/128)*256; for 16-column tile t, 128-row block b, lane
 *   l = 16*kq + j (0 <= j < 16, 0 <= kq < 4) and step u (0 <= u < 4):
 *     tiled[t][256*b + 4*l + u] = gptq[4*(4*b + u) + kq][16*t + j]
 *   with the eight codes of each word reordered: the code of row 8r + i
 *   (bits 4i of the GPTQ word) sits at bits 4*(i/2) + 16*(i%2), i.e. rows
 *   8r, 8r+2, 8r+4, 8r+6 in the low half-word and 8r+1, 8r+3, 8r+5, 8r+7 in
 *   the high one, so that the two codes under one 16-bit mask are
 *   consecutive rows. Words of rows at or beyond K (padding of the last
 *   block) are zero. A row
 *   shard starting at a multiple of 128 rows is the view qweight + 256*(k0/128)
 *   with the same ld_q; a column shard starting at a multiple of 16 columns is
 *   qweight + ld_q*(c0/16). Produced by tpdq_reorder or tpdq_pack_tiled. */
typedef enum { TPDQ_LAYOUT_GPTQ = 0, TPDQ_LAYOUT_TILED = 1 } tpdq_layout;

typedef enum {
  /* Per-row metadata through g_idx (Eq. 3; the naive load of Fig. 1). The
     scale and zero of row k are those of group g_idx[k]; every row looks its
     metadata up separately and the weight is dequantized per element. The
     metadata of a 16-column tile (all num_groups groups) is staged in LDS. */
  TPDQ_PATH_ACTORDER = 0,
  /* Rows sorted by group (Alg. 1; the optimized load of Fig. 2): the group of
     local row k is floor(k / G); g_idx is ignored and may be NULL. With
     group_size 0 (groups of unequal sizes) g_idx is the sorted, non-decreasing
     group index of each row and is required; the rows then take their
     metadata through it (the per-row kernel, on sorted rows). */
  TPDQ_PATH_ORDERED = 1,
  /* As TPDQ_PATH_ACTORDER, but every row fetches its scale and zero from
     global memory (Fig. 1 as drawn, no staging): the baseline for counting
     redundant metadata fetches. */
  TPDQ_PATH_ACTORDER_GLOBAL = 2
} tpdq_path;

/* One quantized layer, or a shard of one given as views (pointer offsets and
 * leading dimensions). K = input features (rows), N = output features.
 * num_groups is the number of metadata rows: ceil(K/G) for a whole or sorted
 * layer; an act-order row-parallel shard keeps the global metadata and global
 * g_idx values, so there num_groups = ceil(K_global/G) exceeds ceil(K/G) (so
 * does a sorted row shard of a layer with groups of unequal sizes, G == 0,
 * whose g_idx then holds its rows' global sorted groups). layout is a
 * tpdq_layout (scales, qzeros and g_idx are always as described above).
 * zero_offset (0 or 1) is added to every stored zero code: 1 for packers that
 * store z - 1 (the zero 16 is then reachable).
 * Alignment: qweight 16 B and ld_q % 4 == 0; scales 8 B and ld_s % 4 == 0;
 * qzeros 4 B; g_idx 16 B. */
typedef struct tpdq_w4 {
  const int32_t* qweight;
  int64_t ld_q;        /* >= N     */
  const void* scales;  /* fp16 (TPDQ_FP16) or bf16 (TPDQ_BF16) */
  int64_t ld_s;        /* >= N     */
  const int32_t* qzeros;
  int64_t ld_z;        /* >= N/8   */
  const int32_t* g_idx;
  int32_t K;
  int32_t N;
  int32_t group_size;  /* G, a multiple of 8; 0: groups of unequal sizes given by g_idx */
  int32_t num_groups;
  int32_t layout;      /* tpdq_layout of qweight */
  int32_t zero_offset; /* 0 or 1, added to each stored zero code */
} tpdq_w4;

/*
 * tpdq_reorder - offline reorder (Alg. 1) and TP-aware fold (section 2.2).
 *
 * For the global (unsharded) layers w1 (K1 x N1) and, optionally, w2
 * (K2 x N2 with K2 == N1), both act-order (g_idx per Eq. 3):
 *   P1 = stable ascending argsort of w1->g_idx, g1_sorted = w1->g_idx[P1];
 *   if w2: P2 = stable argsort of w2->g_idx, g2_sorted = w2->g_idx[P2];
 *   qweight1_out = W1[P1, P2]   (rows gathered by P1, columns by P2;
 *                                without w2 the columns stay in place)
 *   scales1_out  = scales1[:, P2], qzeros1_out = qzeros1[:, P2] (repacked)
 *   qweight2_out = W2[P2]       (rows gathered by P2; scales2 and qzeros2 are
 *                                indexed by group and are reused unchanged)
 * A gather: new index j takes old index P[j]. Ties in the sort keep ascending
 * row order, so P is unique (any stable sort gives the same P).
 *
 * Requirements: every g_idx value in [0, num_groups); with G > 0,
 * num_groups == ceil(K/G) and the groups holding the rows Eq. 3 gives for a
 * permutation phi (G each, the last K - (num_groups - 1) G); with G == 0
 * (groups of unequal sizes) any group sizes. G%8 == 0, N%8 == 0; both inputs
 * in TPDQ_LAYOUT_GPTQ. Outputs are dense:
 * qweight1_out and qweight2_out in out_layout (GPTQ: int32 [K/8][N]; TILED:
 * int32 [ceil(N/16)][ceil(K/128)*256]), scales1_out [num_groups][N1] (the
 * dtype of w1->scales), qzeros1_out int32 [num_groups][N1/8], P and g_sorted
 * int32 [K]. The zero offset of each layer carries over unchanged.
 * P2, g2_sorted and qweight2_out must be NULL when w2 is NULL.
 *
 * Workspace: at least tpdq_workspace_bytes(0, 0, w1, w2) bytes, any content.
 * This call is synchronous in part: it runs the g_idx validation on `stream`
 * and waits for it; on TPDQ_ERR_GIDX nothing has been written to the outputs.
 * After a successful validation the permutation kernels are enqueued and the
 * call returns without waiting for them.
 */
tpdq_status tpdq_reorder(const tpdq_w4* w1, const tpdq_w4* w2,
                         int32_t* P1, int32_t* g1_sorted, int32_t* P2, int32_t* g2_sorted,
                         int32_t* qweight1_out, void* scales1_out, int32_t* qzeros1_out,
                         int32_t* qweight2_out, tpdq_dtype dtype, tpdq_layout out_layout,
                         void* workspace, size_t ws_bytes, void* stream);

/*
 * tpdq_pack_tiled - copy w->qweight (TPDQ_LAYOUT_GPTQ, K x N) into
 * TPDQ_LAYOUT_TILED with ld_q = ceil(K/128)*256: out is int32
 * [ceil(N/16)][ceil(K/128)*256], device, caller-owned. Offline; asynchronous
 * on `stream`. Used to give act-order weights the same storage order as the
 * reordered ones, so that the two GEMM paths differ only in their metadata
 * access (section 2.1, Fig. 1 vs Fig. 2).
 */
tpdq_status tpdq_pack_tiled(const tpdq_w4* w, int32_t* qweight_out, void* stream);

/*
 * tpdq_w4a16_gemm - Y = X' @ deq(W), fp32 accumulation, result rounded to
 * the activation dtype (round to nearest even).
 *
 * X  [M][ldx] activations (K columns used); X' = X, or X[:, x_perm] when
 *    x_perm (int32 [K], device) is given: column j of X' is column x_perm[j]
 *    of X (the X[:, P1] gather of Alg. 2 and Alg. 3); x_perm values outside
 *    [0, K) are clamped. Alignment 16 B and ldx % 8 == 0 (with or without
 *    x_perm: rows are read with 16-byte loads).
 * w  the layer; path selects the metadata load (see tpdq_path). The
 *    act-order paths need w->g_idx; values outside [0, num_groups) are
 *    clamped into range (no fault; such rows give unspecified results).
 * Y  [M][ldy] output, 8 B aligned, ldy % 4 == 0, ldy >= N.
 * Workspace: at least tpdq_workspace_bytes(1, M, w, NULL) bytes, any content
 * (it holds the gathered X' when the gather cannot be done on chip, and the
 * fp32 split-K partials of the kernels that split K: on large weights, and
 * on weights of 16M elements or more when X is row-major and M > 16). A
 * call with x_perm always needs one; without x_perm, a call that needs none
 * accepts NULL. Calls that overlap in time must not share a workspace.
 * Deterministic: the same inputs give bit-identical outputs (split-K
 * partials are added in a fixed order).
 */
tpdq_status tpdq_w4a16_gemm(const void* X, int64_t ldx, int32_t M, const int32_t* x_perm,
                            const tpdq_w4* w, tpdq_path path, tpdq_dtype dtype,
                            void* Y, int64_t ldy,
                            void* workspace, size_t ws_bytes, void* stream);

/*
 * tpdq_mlp_shard - one rank's share of the MLP up to its AllReduce.
 *
 * TPDQ_PATH_ORDERED (Alg. 3): w1 is the rank's column shard of W1[P1, P2],
 *   w2 its row shard of W2[P2] (sorted rows, so local groups are floor(k/G));
 *   Y1 = X[:, P1] @ deq(w1), Y2_partial = Y1 @ deq(w2). No permute or gather
 *   of Y1 happens between the GEMMs. P1 (int32 [K1], global) is required.
 * TPDQ_PATH_ACTORDER / TPDQ_PATH_ACTORDER_GLOBAL: w1 is the rank's column
 *   shard of W1 with its g_idx, w2 the row shard of W2 with its rows' global
 *   g_idx values and the full metadata (num_groups = K2_global/G); P1 must be
 *   NULL.
 * Requirements: w2->K == w1->N. X [M][ldx] with w1->K columns used, 16-byte
 * aligned, ldx % 8 == 0 (on every path).
 * Y1 [M][w1->N] and Y2_partial [M][w2->N], dense, written in the activation
 * dtype; Y2_partial is this rank's summand of the AllReduce(SUM) of Alg. 3.
 * Workspace: tpdq_workspace_bytes(2, M, w1, w2) bytes, any content.
 */
tpdq_status tpdq_mlp_shard(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                           const tpdq_w4* w1, const tpdq_w4* w2, tpdq_path path,
                           tpdq_dtype dtype, void* Y1, void* Y2_partial,
                           void* workspace, size_t ws_bytes, void* stream);

/*
 * tpdq_mlp_shard_noalloc - tpdq_mlp_shard for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same computation, kernels and results, without a
 * workspace argument. The workspace is a static scratch array of 64 MiB that
 * the library holds on each GPU it runs on until the process ends; this call
 * never allocates or frees device memory and calls no allocating routine.
 * Arguments, alignment and results as for tpdq_mlp_shard; the scratch serves
 * the stream's device. A call whose tpdq_workspace_bytes(2, M, w1, w2) exceeds
 * 64 MiB returns TPDQ_ERR_WORKSPACE before any device work (every decode and
 * prefill shape of the paper's workloads fits; e.g. M = 2048 on the Llama-70B
 * TP = 2 shard uses 32 MiB). The scratch needs no particular content. All
 * calls on one GPU share its scratch: calls that overlap in time on one GPU
 * (two streams, two threads) race and must be serialised by the caller. The
 * first call on a device resolves that device's scratch address (a runtime
 * symbol lookup, no allocation).
 */
tpdq_status tpdq_mlp_shard_noalloc(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                                   const tpdq_w4* w1, const tpdq_w4* w2, tpdq_path path,
                                   tpdq_dtype dtype, void* Y1, void* Y2_partial, void* stream);

/*
 * tpdq_gated_mlp_shard - one rank's share of an MLP with a gate projection,
 * up to its AllReduce: Y1 = silu(X' W_gate) * (X' W_up) (silu(x) =
 * x / (1 + e^-x), both products in fp32, one rounding), Y2_partial = Y1 @
 * W_down. The experiments section notes that the method carries over to
 * this MLP: P2 (from W_down) is folded into the columns of both W_gate and
 * W_up, since the elementwise silu(gate) * up commutes with a column
 * permutation.
 *
 * Gate and up take the same input, so act-order gives them one permutation:
 * TPDQ_PATH_ORDERED: w_gate and w_up are the rank's column shards of
 *   W_gate[P1, P2] and W_up[P1, P2] (tpdq_reorder(w_gate, w_down) and
 *   tpdq_reorder(w_up, w_down) give the same P1 when their g_idx agree),
 *   w_down its row shard of W_down[P2]; X' = X[:, P1], P1 required.
 * TPDQ_PATH_ACTORDER / TPDQ_PATH_ACTORDER_GLOBAL: w_gate, w_up and w_down as
 *   for tpdq_mlp_shard; w_gate->g_idx serves both gate and up (w_up->g_idx
 *   is not read); P1 must be NULL.
 * w_up must have w_gate's K, N, group size, num_groups, layout, leading
 * dimensions and zero offset (TPDQ_ERR_SHAPE otherwise); w_down->K == w_gate->N.
 * X, Y1, Y2_partial, alignment and workspace as for tpdq_mlp_shard, with
 * tpdq_workspace_bytes(3, M, w_gate, w_down). Runs the decode kernels at
 * every M (batches of more than 64 rows in launches of 64).
 */
tpdq_status tpdq_gated_mlp_shard(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                                 const tpdq_w4* w_gate, const tpdq_w4* w_up, const tpdq_w4* w_down,
                                 tpdq_path path, tpdq_dtype dtype, void* Y1, void* Y2_partial,
                                 void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes for op 0 (tpdq_reorder: a = w1, b = w2 or NULL),
 * 1 (tpdq_w4a16_gemm: a = w), 2 (tpdq_mlp_shard: a = w1, b = w2) or
 * 3 (tpdq_gated_mlp_shard: a = w_gate, b = w_down) at batch M. Returns 0
 * when the arguments are invalid. */
size_t tpdq_workspace_bytes(int op, int32_t M, const tpdq_w4* a, const tpdq_w4* b);

/* Static description of a status code. */
const char* tpdq_status_string(tpdq_status s);

/* Detail of the last non-OK status returned on the calling thread. */
const char* tpdq_last_error(void);

/* Library version, e.g. "0.1.0". */
const char* tpdq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TPDQ_H */
