/*
 * lorex.h -- C ABI of the LorExperts / BTExperts MoE-layer forward for MI355X.
 *
 * The operation (arXiv 2608.07814):
 *   Sec. 3 "Representation": the E experts of one MoE layer are partitioned
 *   into clusters; each cluster keeps one full-precision dominant expert and
 *   every other member m is stored as a rank-r correction of it, per
 *   projection:  W_m = W_dom + A_m B_m  (A output-side, B input-side).
 *   Sec. 5 / Fig. tree (BTExperts): anchors and corrections may be nested in a
 *   tree whose leaves are the experts; an expert's weights are the anchor plus
 *   the corrections of every node on its path.
 *   The router is unchanged (Fig. overview): top-k ids and weights are inputs.
 *   Expert FFN: y = W_down (silu(W_gate x) * (W_up x)), no biases.
 *   out[t] = sum_j topk_weights[t][j] * y_{topk_ids[t][j]}(x_t).
 *   Sec. 5.1 "Amortized forward pass": terms shared by co-selected experts are
 *   computed once per token; the library applies each anchor's gate/up once
 *   per (token, anchor), each node's correction once per (token, node), and by
 *   linearity each down projection once to the routing-weighted sum of the
 *   activations below it.
 *
 * Conventions for every entry point:
 *   - All array arguments are DEVICE pointers to caller-owned memory (the
 *     layer descriptor structs themselves live on the host and are read during
 *     the call only). The library never allocates or frees device memory and
 *     keeps no pointer past the call. The only resources it creates itself are
 *     described under "Auxiliary stream" below.
 *   - Weights use nn.Linear layout [out][in], input dimension contiguous.
 *     Every array is dense row-major; pointers must be 16-byte aligned.
 *   - x and all weights share one dtype (LX_BF16 or LX_F32). bf16 inputs are
 *     multiplied with fp32 accumulation; fp32 inputs use fp32 arithmetic.
 *     d and f must be multiples of 8 (LX_ERR_UNSUPPORTED otherwise), and so
 *     must every correction rank of a bf16 layer.
 *   - topk_ids [T][k] int32: -1 marks a dropped slot (contributes nothing);
 *     an id < -1 or >= E is invalid: it is dropped and LX_DEVFLAG_BAD_ID is
 *     raised in the workspace (read it with lx_read_device_status). Duplicate
 *     ids in a row are legal and act as independent slots.
 *   - topk_weights [T][k] fp32 are used as given (never renormalized).
 *   - out [T][d] is fully overwritten (LX_F32 or LX_BF16).
 *   - `workspace` is device memory of at least the size the matching
 *     *_workspace_bytes function returns; its contents need no initialization.
 *   - `stream` is a hipStream_t (NULL = the default stream). Every call is
 *     asynchronous on that stream; inputs must stay valid until the stream's
 *     work completes. Calls with distinct workspaces may be issued from
 *     several host threads at once (see the serialisation noted below).
 *   - T = 0 is a valid no-op. Host-side argument errors are returned before
 *     anything is enqueued; the message is available from lx_last_error().
 *
 * Auxiliary stream (forward entry points only; off unless enabled with
 * lx_set_aux_stream(1): every large GEMM is a persistent kernel holding one
 * workgroup per compute unit, so two chains mostly take turns, and the
 * measured forwards run slightly faster on one stream). When enabled, a
 * batch is large enough for the anchor GEMMs to run on the persistent
 * large-tile kernel and the layer has corrections, the correction GEMM
 * chains are forked onto a second
 * stream of the same device (default priority, non-blocking) between two
 * events recorded on the caller's stream, so they overlap the anchor GEMMs;
 * the caller's stream is ordered after all of the call's work when the call
 * returns. That stream and its two events are created on the first such call
 * on each device and kept until the process ends (per device, shared by all
 * callers). A per-device mutex is held while a forward enqueues its work
 * (host side only), so concurrent forwards on one device enqueue one after
 * another, and their correction chains run one after another on the shared
 * stream. With it off (the default) every launch goes to the caller's
 * stream, nothing is created and no lock is taken. Decode-sized
 * batches and per-kernel timing (lx_profile_enable) never use it. Mutable
 * global state besides this: the switch itself, the per-thread error message
 * and the optional kernel-timing records.
 */
#ifndef LOREX_H
#define LOREX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lx_status {
  LX_OK = 0,
  LX_ERR_INVALID_ARGUMENT = 1,   /* null/misaligned pointer, bad size or count */
  LX_ERR_UNSUPPORTED = 2,        /* valid but not implemented (e.g. d % 8 != 0 in bf16) */
  LX_ERR_WORKSPACE_TOO_SMALL = 3,
  LX_ERR_HIP = 4                 /* a HIP runtime call failed */
} lx_status;

typedef enum lx_dtype { LX_F32 = 0, LX_BF16 = 1 } lx_dtype;

#define LX_MAX_LEVELS 4      /* correction levels below the anchors */
#define LX_MAX_K 32          /* largest supported top-k */
#define LX_MAX_NODES 8192    /* largest node count of any level (incl. E) */

/* Device-side status bits, accumulated in the workspace by each call. */
#define LX_DEVFLAG_BAD_ID 1u     /* a topk id < -1 or >= E (slot dropped) */
#define LX_DEVFLAG_BAD_TREE 2u   /* a parent or factor index out of range
                                    (the node's expert slots are dropped or the
                                    correction ignored) */

/* One correction level of a tree (Sec. 5, Fig. tree). Node i of this level is
 * its parent's weights plus, when factor_of[i] >= 0, the rank-`rank` product
 * of factor pair factor_of[i]:
 *   gate: A_gate[m] (f x rank) * B_gate[m] (rank x d)
 *   up:   A_up[m]   (f x rank) * B_up[m]   (rank x d)
 *   down: A_down[m] (d x rank) * B_down[m] (rank x f)            */
typedef struct lx_level {
  int32_t n_nodes;           /* nodes of this level */
  int32_t rank;              /* rank of its corrections (multiple of 8 for bf16) */
  int32_t n_factors;         /* factor pairs stored */
  const int32_t* parent;     /* [n_nodes] node index one level up */
  const int32_t* factor_of;  /* [n_nodes] factor pair index, or -1 (no correction) */
  const void* a_gate;        /* [n_factors][f][rank] */
  const void* b_gate;        /* [n_factors][rank][d] */
  const void* a_up;          /* [n_factors][f][rank] */
  const void* b_up;          /* [n_factors][rank][d] */
  const void* a_down;        /* [n_factors][d][rank] */
  const void* b_down;        /* [n_factors][rank][f] */
  /* Optional (NULL = not used, all four or none): fp16 copies of the factors
   * made by lx_convert_f16 (one power-of-two scale per factor matrix). With
   * them, batches on the fp16 anchor path (see lx_convert_f16) run every
   * correction product of the level as one fp16 product: the rank-`rank`
   * intermediates and the level's activation sums are fp16 with power-of-two
   * scales instead of bf16 (hi, lo) pairs. */
  const void* a_gate_f16;            /* [n_factors][f][rank] */
  const int32_t* a_gate_f16_exp;     /* [n_factors] */
  const void* a_up_f16;              /* [n_factors][f][rank] */
  const int32_t* a_up_f16_exp;       /* [n_factors] */
  const void* a_down_f16;            /* [n_factors][d][rank] */
  const int32_t* a_down_f16_exp;     /* [n_factors] */
  const void* b_down_f16;            /* [n_factors][rank][f] */
  const int32_t* b_down_f16_exp;     /* [n_factors] */
  /* Padded rank of the fp16 copies (0: rank). The fp16 path needs the rank
   * to be a multiple of 64; for another rank the copies can be made at
   * rank_f16 = rank rounded up to a multiple of 64 (lx_convert_f16_padded),
   * with zero columns (a_*_f16: [n_factors][f or d][rank_f16]) or zero rows
   * (b_down_f16: [n_factors][rank_f16][f]) beyond rank, together with bf16
   * copies of b_gate and b_up padded with zero rows (lx_pad_bf16). The
   * padding holds exact zeros, so the products equal those of rank `rank`.
   * rank_f16 > rank requires both pad copies; at most 128. */
  int32_t rank_f16;
  const void* b_gate_pad;            /* [n_factors][rank_f16][d] bf16 */
  const void* b_up_pad;              /* [n_factors][rank_f16][d] bf16 */
} lx_level;

/* A BTExperts tree (Sec. 5): dense anchors, then n_levels correction levels;
 * the nodes of the last level are the E experts (levels[n_levels-1].n_nodes
 * must equal E; with n_levels = 0 the anchors are the experts). */
typedef struct lx_tree_layer {
  int32_t E, d, f;
  lx_dtype dtype;
  int32_t n_anchors;
  const void* anchor_gate;   /* [n_anchors][f][d] */
  const void* anchor_up;     /* [n_anchors][f][d] */
  const void* anchor_down;   /* [n_anchors][d][f] */
  int32_t n_levels;          /* 0 .. LX_MAX_LEVELS */
  lx_level levels[LX_MAX_LEVELS];
  /* Optional (NULL = not used): fp8 copy of anchor_down made by
   * lx_quantize_f8. With it the anchor down projection multiplies the low
   * half of its bf16 (hi, lo) input split in fp8 (see lx_quantize_f8). */
  const void* anchor_down_f8;            /* [n_anchors][d][f] e4m3 */
  const uint32_t* anchor_down_f8_scale;  /* [n_anchors][d][f / 64] */
  /* Optional (NULL = not used): fp16 copy of anchor_down made by
   * lx_convert_f16. With it, batches whose activation sums fit the fp16 path
   * (see lx_convert_f16) run the anchor down projection as one fp16 product
   * instead of the bf16 (hi, lo) pair; it takes precedence over the fp8 copy. */
  const void* anchor_down_f16;           /* [n_anchors][d][f] fp16, scaled */
  const int32_t* anchor_down_f16_exp;    /* [n_anchors] scale exponents */
} lx_tree_layer;

/* A flat LorExperts layer (Sec. 3 "Representation"): C clusters, one dominant
 * per cluster, members W_dom + A B with rank r. Equivalent to a tree with one
 * correction level whose parent map is cluster_of. */
typedef struct lx_flat_layer {
  int32_t E, C, d, f, r, M;  /* experts, clusters, hidden, intermediate, rank, factor pairs */
  lx_dtype dtype;
  const int32_t* cluster_of; /* [E] cluster of each expert */
  const int32_t* factor_of;  /* [E] factor pair of each expert, -1 for a dominant */
  const void* dom_gate;      /* [C][f][d] */
  const void* dom_up;        /* [C][f][d] */
  const void* dom_down;      /* [C][d][f] */
  const void* a_gate;        /* [M][f][r] */
  const void* b_gate;        /* [M][r][d] */
  const void* a_up;          /* [M][f][r] */
  const void* b_up;          /* [M][r][d] */
  const void* a_down;        /* [M][d][r] */
  const void* b_down;        /* [M][r][f] */
  const void* dom_down_f8;             /* optional fp8 copy of dom_down (lx_quantize_f8) */
  const uint32_t* dom_down_f8_scale;   /* its scale words, [C][d][f / 64] */
  const void* dom_down_f16;            /* optional fp16 copy of dom_down (lx_convert_f16) */
  const int32_t* dom_down_f16_exp;     /* its scale exponents, [C] */
  /* optional fp16 copies of the factors (lx_convert_f16; all four or none),
   * as the fp16 factor copies of lx_level */
  const void* a_gate_f16;
  const int32_t* a_gate_f16_exp;       /* [M] */
  const void* a_up_f16;
  const int32_t* a_up_f16_exp;
  const void* a_down_f16;
  const int32_t* a_down_f16_exp;
  const void* b_down_f16;
  const int32_t* b_down_f16_exp;
  /* padded rank of the fp16 copies and the padded bf16 copies of b_gate and
   * b_up, as rank_f16, b_gate_pad and b_up_pad of lx_level */
  int32_t r_f16;
  const void* b_gate_pad;              /* [M][r_f16][d] */
  const void* b_up_pad;                /* [M][r_f16][d] */
} lx_flat_layer;

/* An uncompressed MoE layer (every expert stored in full): the comparator the
 * compressed layers are measured against, computed with the same kernels and
 * precision policy. */
typedef struct lx_dense_layer {
  int32_t E, d, f;
  lx_dtype dtype;
  const void* w_gate;        /* [E][f][d] */
  const void* w_up;          /* [E][f][d] */
  const void* w_down;        /* [E][d][f] */
  const void* w_down_f8;               /* optional fp8 copy of w_down (lx_quantize_f8) */
  const uint32_t* w_down_f8_scale;     /* its scale words, [E][d][f / 64] */
  const void* w_down_f16;              /* optional fp16 copy of w_down (lx_convert_f16) */
  const int32_t* w_down_f16_exp;       /* its scale exponents, [E] */
} lx_dense_layer;

/* Human-readable name of a status code (static string). */
const char* lx_status_string(lx_status s);
/* Message of the last failed call on this thread ("" if none). */
const char* lx_last_error(void);
/* Library version, major*10000 + minor*100 + patch. */
int32_t lx_version(void);

/* Workspace bytes needed by one forward call with T tokens and top-k k.
 * Returns 0 and sets lx_last_error() if the descriptor or sizes are invalid
 * (only sizes and counts are inspected; no device memory is read). */
size_t lx_moe_workspace_bytes(const lx_flat_layer* layer, int32_t T, int32_t k);
size_t lx_moe_tree_workspace_bytes(const lx_tree_layer* layer, int32_t T, int32_t k);
size_t lx_dense_moe_workspace_bytes(const lx_dense_layer* layer, int32_t T, int32_t k);

/* Flat LorExperts forward (Sec. 3 representation, Sec. 5.1 amortization).
 * x [T][d] (layer dtype); out [T][d] (out_dtype). */
lx_status lx_moe_forward(const lx_flat_layer* layer, int32_t T, int32_t k,
                         const void* x, const int32_t* topk_ids,
                         const float* topk_weights, void* out, lx_dtype out_dtype,
                         void* workspace, size_t workspace_bytes, void* stream);

/* BTExperts tree forward (Sec. 5); same arguments as lx_moe_forward. */
lx_status lx_moe_forward_tree(const lx_tree_layer* layer, int32_t T, int32_t k,
                              const void* x, const int32_t* topk_ids,
                              const float* topk_weights, void* out, lx_dtype out_dtype,
                              void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the tree
 * forward of lx_moe_forward_tree with the same arguments minus the
 * workspace, which is replaced by a library-owned static device array of
 * LX_STATIC_SCRATCH_BYTES (64 MiB) per GPU, created when the library's code
 * is loaded on that GPU and held until the process ends. The call allocates
 * nothing and creates no HIP object: no hipMalloc/hipFree, no auxiliary
 * stream (every launch goes to `stream`), no kernel-timing records; the
 * first call on a device looks the array's device address up once.
 * A batch whose workspace (lx_moe_tree_workspace_bytes) exceeds the array is
 * refused with LX_ERR_WORKSPACE_TOO_SMALL before anything is enqueued; 64 MiB
 * covers decode-sized batches (e.g. T <= 64 at d = 4096, f = 1024 with two
 * correction levels; T <= 128 at d = 2048, f = 768, 128 experts, top-8).
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind; the forward initialises everything it reads, so nothing needs
 * clearing. Calls whose device work overlaps on one GPU (several host threads
 * or streams at once) race on the array: serialise them. The device status
 * word (LX_DEVFLAG_*) lives in the array and is not exposed: an invalid id is
 * dropped silently. Flat layers are passed as their one-level tree. */
#define LX_STATIC_SCRATCH_BYTES (64u << 20)
lx_status lx_moe_forward_tree_static(const lx_tree_layer* layer, int32_t T, int32_t k,
                                     const void* x, const int32_t* topk_ids,
                                     const float* topk_weights, void* out, lx_dtype out_dtype,
                                     void* stream);

/* Uncompressed top-k SwiGLU MoE (comparator); same arguments. */
lx_status lx_dense_moe_forward(const lx_dense_layer* layer, int32_t T, int32_t k,
                               const void* x, const int32_t* topk_ids,
                               const float* topk_weights, void* out, lx_dtype out_dtype,
                               void* workspace, size_t workspace_bytes, void* stream);

/* fp8 copy of bf16 weights, for the anchor down projection.
 *
 * The precision policy keeps every fp32 intermediate that feeds a bf16 GEMM
 * as a bf16 (hi, lo) pair, and the GEMM runs K twice: C = (hi + lo) W^T. The
 * lo half is below 2^-8 of hi, so a few bits of it suffice: given an fp8 copy
 * of the anchor down weights (layer field anchor_down_f8 / dom_down_f8 /
 * w_down_f8 and its scale words), the anchor activation sums are stored as
 * bf16 hi plus a block-scaled fp8 lo, and lo W^T runs on the gfx950
 * block-scaled fp8 MFMA at twice the bf16 rate with half the bytes. Used for
 * batches large enough for the large-tile kernel; decode-sized batches keep
 * the bf16 pair.
 *
 * w [n][rows][cols] bf16 -> w_f8 [n][rows][cols] OCP e4m3 bytes (round to
 * nearest even) and scales [n][rows][cols / 64] uint32: bytes 0 and 1 are the
 * E8M0 exponents (value 2^(byte - 127)) of the two 32-column blocks of each
 * 64-column slab, chosen so that each block's largest magnitude maps into
 * [128, 256); bytes 2 and 3 are zero. cols must be a multiple of 64
 * (LX_ERR_UNSUPPORTED otherwise); w_f8 16-byte and scales 4-byte aligned.
 * Asynchronous on `stream`. */
lx_status lx_quantize_f8(const void* w, int32_t n, int32_t rows, int32_t cols, void* w_f8,
                         uint32_t* scales, void* stream);

/* fp16 copy of bf16 weights, for the anchor down projection and the
 * correction products.
 *
 * The anchor down projection multiplies the anchor activation sums hbar
 * (Sec. 5.1: the routing-weighted sum of the SwiGLU activations of a token's
 * experts under one anchor) by the anchor's down weights. Rounded to bf16,
 * hbar costs about 1e-2 x RMS of the output (the acceptance bar), hence the
 * (hi, lo) pair; fp16 keeps 3 more bits (about 1.3e-3 x RMS) at the bf16 MFMA
 * rate in a single product. With this copy in the layer, the forward stores
 * hbar as fp16 with one power-of-two scale per token (the largest magnitude
 * over the token's fp16 sums in [2^14, 2^15)) and multiplies it with the
 * copy, undoing both scales exactly in the output. Used for batches of at
 * least 512 tokens with f a multiple of 256 and at most 1024, k <= 8 and at
 * most two correction levels, on the large-tile kernel; other batches take
 * the fp8 copy (if any) or the pair. With fp16 copies of a level's factors
 * too (lx_level), that level's correction products run the same way: its
 * activation sums as above, its rank-r intermediates fp16 with one
 * power-of-two scale per 256-row tile (rank a multiple of 64, at most 128, or
 * copies padded to such a rank: lx_convert_f16_padded; levels with at most 64
 * rows per node keep the pair).
 *
 * w [n][rows][cols] bf16 -> w_f16 [n][rows][cols] fp16 equal to w * 2^e_i
 * for matrix i, rounded to nearest even, with exps[i] = e_i chosen so that
 * the matrix's largest magnitude lands in [2^14, 2^15) (0 for an all-zero
 * matrix); exact for every bf16 value down to 2^-28 of that maximum. Device
 * pointers: w_f16 16-byte aligned, exps 4-byte aligned; n, rows, cols >= 1
 * (LX_ERR_INVALID_ARGUMENT). Asynchronous on `stream`. */
lx_status lx_convert_f16(const void* w, int32_t n, int32_t rows, int32_t cols, void* w_f16, int32_t* exps,
                         void* stream);

/* lx_convert_f16 into a larger zero-padded layout, for the factor copies of
 * a level whose rank is not a multiple of 64 (lx_level::rank_f16).
 *
 * w [n][rows][cols] bf16 -> w_f16 [n][rows_out][cols_out] fp16: element
 * (i, r, c) is w[i][r][c] * 2^exps[i] for r < rows and c < cols (the same
 * values and exponents as lx_convert_f16) and 0 elsewhere. rows_out >= rows,
 * cols_out >= cols, all positive (LX_ERR_INVALID_ARGUMENT); pointers as in
 * lx_convert_f16. Asynchronous on `stream`. */
lx_status lx_convert_f16_padded(const void* w, int32_t n, int32_t rows, int32_t cols, int32_t rows_out,
                                int32_t cols_out, void* w_f16, int32_t* exps, void* stream);

/* Zero-padded bf16 copy (the padded b_gate and b_up of lx_level::rank_f16):
 * w [n][rows][cols] bf16 -> w_out [n][rows_out][cols_out] bf16, element
 * (i, r, c) = w[i][r][c] for r < rows and c < cols, 0 elsewhere. rows_out >=
 * rows, cols_out >= cols, all positive (LX_ERR_INVALID_ARGUMENT); w_out
 * 16-byte aligned. Asynchronous on `stream`. */
lx_status lx_pad_bf16(const void* w, int32_t n, int32_t rows, int32_t cols, int32_t rows_out, int32_t cols_out,
                      void* w_out, void* stream);

/* The model's unchanged top-k router on the GPU (Sec. 3 "Stage 1" and Fig.
 * overview: compression leaves the router as it is and every expert
 * addressable), producing the routing inputs of lx_moe_forward /
 * lx_moe_forward_tree / lx_dense_moe_forward on the same stream, with no
 * host round trip.
 *
 * logits[t][e] = sum_i w_r[e][i] * x[t][i] (fp32 accumulation of the exact
 * bf16 products); topk_ids[t][0..k) = the k largest logits in descending
 * order, equal logits ordered by ascending expert index (NaN below every
 * number); topk_weights[t][j] = exp(l_j - l_0) / sum_i exp(l_i - l_0) over the
 * chosen logits (the softmax over all E restricted to the chosen experts and
 * renormalised to sum 1).
 *
 * x [T][d] and w_r [E][d] bf16 (dtype must be LX_BF16, else
 * LX_ERR_UNSUPPORTED), 16-byte aligned; topk_ids [T][k] int32 and
 * topk_weights [T][k] fp32, 4-byte aligned, caller-owned, fully overwritten;
 * workspace 256-byte aligned, at least lx_route_workspace_bytes(T, d, E)
 * bytes (LX_ERR_WORKSPACE_TOO_SMALL), contents irrelevant on entry. d a
 * positive multiple of 64, E a multiple of 4 in 4 .. 512, T * d < 2^31
 * (LX_ERR_UNSUPPORTED); 1 <= k <= min(E, LX_MAX_K) (LX_ERR_INVALID_ARGUMENT).
 * T = 0 is a no-op. Deterministic run to run. Asynchronous on `stream`. */
size_t lx_route_workspace_bytes(int32_t T, int32_t d, int32_t E);
lx_status lx_route_topk(const void* x, const void* w_r, lx_dtype dtype, int32_t T, int32_t d, int32_t E,
                        int32_t k, int32_t* topk_ids, float* topk_weights, void* workspace,
                        size_t workspace_bytes, void* stream);

/* The unchanged router fused into the tree forward (Sec. 3 "Stage 1" and
 * Fig. overview: the router is left as it is and selects among all experts;
 * Sec. 5.1: the forward shares work among the experts it selects). The
 * router's logits x W_r^T run first (as in lx_route_topk); their top-k and
 * renormalised softmax are computed inside the first bucketing kernel, which
 * writes topk_ids and topk_weights (outputs here, same values and layout as
 * lx_route_topk's, bit for bit) and organises them into the rows the forward
 * shares, so routing and bucketing take one launch fewer than
 * lx_route_topk followed by lx_moe_forward_tree. Batches of at most 64
 * tokens, whose bucketing is a single workgroup, keep the router's own top-k
 * launch (one workgroup would take every token's top-k on one compute
 * unit). Then the forward as lx_moe_forward_tree on those ids and weights:
 * out is bitwise the same.
 *
 * layer: as for lx_moe_forward_tree, bf16 (LX_ERR_UNSUPPORTED otherwise);
 * w_r [E][d] bf16, 16-byte aligned; E a multiple of 4 in 4 .. 512, k <=
 * min(E, LX_MAX_K) (as lx_route_topk); topk_ids [T][k] int32 and
 * topk_weights [T][k] fp32, caller-owned device memory, fully overwritten;
 * workspace 256-byte aligned, lx_route_moe_tree_workspace_bytes(layer, T, k)
 * bytes (0 for an invalid or unsupported call). Asynchronous on `stream`;
 * the auxiliary-stream conventions of the forward apply. */
size_t lx_route_moe_tree_workspace_bytes(const lx_tree_layer* layer, int32_t T, int32_t k);
lx_status lx_route_moe_forward_tree(const lx_tree_layer* layer, int32_t T, int32_t k, const void* x,
                                    const void* w_r, int32_t* topk_ids, float* topk_weights, void* out,
                                    lx_dtype out_dtype, void* workspace, size_t workspace_bytes, void* stream);

/* Router profiling and the Coact-NPMI clustering distance (Sec. 3,
 * "Compression pipeline", Stage 1, and "Variants"), from the routing ids of N
 * calibration tokens (topk_ids [N][k] int32, device; ids outside [0, E) and
 * repeated ids within a row are ignored).
 *
 * fire [E] uint32: tokens on which expert e fires; pair [E][E] uint32
 * (symmetric, zero diagonal): tokens on which both fire; dist [E][E] fp64:
 * D = 1 - NPMI with p_i = fire[i] / N, p_ij = pair[i][j] / N, NPMI = log(p_ij /
 * (p_i p_j)) / (-log p_ij), NPMI = -1 for pairs that never co-fire and 1 for
 * pairs that co-fire on every token, zero diagonal. All outputs caller-owned
 * device memory (4-, 4- and 8-byte aligned), fully overwritten. E in 1 ..
 * 1024 (LX_ERR_UNSUPPORTED), 1 <= k <= LX_MAX_K and N >= 0
 * (LX_ERR_INVALID_ARGUMENT). Exact integer counts; asynchronous on `stream`. */
lx_status lx_coact_distance(const int32_t* topk_ids, int32_t N, int32_t k, int32_t E, uint32_t* fire,
                            uint32_t* pair, double* dist, void* stream);

/* Frequency-seeded k-medoids and the dominant choice (Sec. 3, Stage 2):
 * clusters C experts' worth of medoids over the distance dist [E][E] fp64
 * (device; any symmetric matrix with zero diagonal, e.g. lx_coact_distance's)
 * and firing counts fire [E] uint32 (device).
 *
 * The experts listed in protected_ids (HOST array, n_protected distinct ids)
 * become singleton clusters C - n_protected .. C - 1 in ascending id order.
 * The others: seeds = the C - n_protected highest-firing ones (ties: lower
 * id), cluster c seeded by the c-th; then assign (nearest medoid, ties to the
 * lower cluster; a medoid stays in its own cluster) and update (the member
 * with the smallest sum of distances to its cluster, summed in ascending
 * member order; ties: lower id) until no medoid changes, at most max_iter
 * updates. Dominant of a cluster: highest firing count, then the largest sum
 * of (1 - dist) to the other members, then the lower id.
 *
 * Outputs (device, caller-owned): cluster_of [E] and factor_of [E] int32 in
 * the layout lx_flat_layer takes (factor_of = -1 for a dominant, 0, 1, ...
 * for the other experts in ascending id order), dominant [C] int32,
 * iterations [1] int32 (update rounds run). E in 1 .. 1024
 * (LX_ERR_UNSUPPORTED); 1 <= C - n_protected <= E - n_protected, ids in range
 * and distinct, max_iter >= 0 (LX_ERR_INVALID_ARGUMENT). Decisions are exact
 * fp64 comparisons: deterministic. Asynchronous on `stream`. */
lx_status lx_kmedoids(const double* dist, const uint32_t* fire, int32_t E, int32_t C, const int32_t* protected_ids,
                      int32_t n_protected, int32_t max_iter, int32_t* cluster_of, int32_t* factor_of,
                      int32_t* dominant, int32_t* iterations, void* stream);

/* Stage 3, neuron alignment (Sec. 3, "Alignment and low-rank decomposition"
 * (i), eqs. cost and assign). Neuron i of an expert is the concatenation of
 * gate row i, up row i and down column i (3d values); the cost of matching
 * the dominant's neuron i with the member's neuron j is
 * cost[i][j] = ||a_i||^2 + ||b_j||^2 - 2 a_i . b_j, computed in fp64 from the
 * stored weights (gate, up [f][d], down [d][f], LX_BF16 or LX_F32, device,
 * element-aligned). cost [f][f] fp64 device (8-byte aligned); workspace
 * 256-byte aligned, lx_align_workspace_bytes(f, d) bytes
 * (LX_ERR_WORKSPACE_TOO_SMALL). f * 3d < 2^31 (LX_ERR_UNSUPPORTED).
 * Asynchronous on `stream`. */
size_t lx_align_workspace_bytes(int32_t f, int32_t d);
lx_status lx_align_cost(const void* dom_gate, const void* dom_up, const void* dom_down, const void* mem_gate,
                        const void* mem_up, const void* mem_down, lx_dtype dtype, int32_t f, int32_t d, double* cost,
                        void* workspace, size_t workspace_bytes, void* stream);

/* The exact minimum-cost perfect matching of an n x n cost matrix (eq.
 * assign), on the HOST: cost [n][n] fp64 host memory; perm [n] int32 host
 * memory receives, for each row i, the column matched to it; total (may be
 * NULL) its summed cost. Shortest augmenting paths with dual potentials (the
 * augmentation phase of Jonker-Volgenant), O(n^3). Synchronous; no GPU. */
lx_status lx_assign(const double* cost, int32_t n, int32_t* perm, double* total);

/* Stage 3, low-rank factors (eqs. svd and factors): the rank-r truncated SVD
 * of the aligned residual R = W_m^P - W_dom (rows x cols; the member's rows,
 * perm_axis 0, or columns, perm_axis 1, taken in the order perm [device
 * int32, or NULL for none]) from a randomized solver, split symmetrically:
 * A = U_r Sigma_r^(1/2) [rows][r] and B = Sigma_r^(1/2) V_r^T [r][cols] fp32
 * (output-side and input-side factors of W ~ W_dom + A B), sigma [r] fp64.
 * Solver: subspace iteration with the Gaussian test matrix omega
 * [cols][r + p] fp64 (device, caller-drawn), q power iterations, every
 * product orthonormalised (CholeskyQR2), then the eigendecomposition of the
 * small Gram matrix of Q^T R (cyclic Jacobi). All in fp64. A sketch
 * direction the residual does not have (exactly low-rank R) yields a zero
 * basis column and carries no weight.
 *
 * w_dom, w_mem [rows][cols] LX_BF16 or LX_F32 (device); r >= 1, p >= 0,
 * 0 <= q <= 16 (LX_ERR_INVALID_ARGUMENT); r + p <= min(128, rows, cols),
 * rows * cols < 2^31 (LX_ERR_UNSUPPORTED); workspace 256-byte aligned,
 * lx_lowrank_workspace_bytes(rows, cols, r, p) bytes. Asynchronous on
 * `stream`; deterministic. */
size_t lx_lowrank_workspace_bytes(int32_t rows, int32_t cols, int32_t r, int32_t p);
lx_status lx_lowrank_factors(const void* w_dom, const void* w_mem, lx_dtype dtype, int32_t rows, int32_t cols,
                             const int32_t* perm, int32_t perm_axis, int32_t r, int32_t p, int32_t q,
                             const double* omega, float* A, float* B, double* sigma, void* workspace,
                             size_t workspace_bytes, void* stream);

/* Stage 3, activation-weighted factors (the output-matching objective of
 * Sec. 4, reconstruction fine-tuning; its closed form, whitening by the
 * activation second moment and one SVD, in Secs. 6 "Calibration cost" and
 * 7 "Hessian-weighted fitting"): the rank-r (A, B) minimising the error the
 * member emits on calibration activations x [n][cols] (one token per row),
 *   ||(R - A B) x^T||_F^2 + damp ||R - A B||_F^2,
 * for the aligned residual R as in lx_lowrank_factors. With G = x^T x +
 * damp I = L L^T the optimum is the rank-r truncation of R L = U S V^T:
 * A = U_r S_r^(1/2) [rows][r], B = S_r^(1/2) V_r^T L^(-1) = S_r^(-1/2)
 * U_r^T R [r][cols] fp32, sigma = S_r [r] fp64 (rows of B and columns of A
 * with sigma = 0 are 0). damp >= 0 is a ridge term for experts that saw few
 * tokens (with damp = 0 and x not of full column rank the optimum is not
 * unique; this returns the one with B in the row space of U_r^T R).
 * Solver: lx_lowrank_factors' randomized subspace iteration applied to the
 * operator M = R x'^T, x' = [x; sqrt(damp) I] (M M^T = R G R^T: the left
 * singular vectors and values of R L), with the caller's Gaussian test
 * matrix omega [n'][r + p] fp64 (device), n' = n + (damp > 0 ? cols : 0).
 *
 * w_dom, w_mem [rows][cols] LX_BF16 or LX_F32 (device); x [n][cols] LX_BF16
 * or LX_F32 (device, may be NULL when n = 0); r >= 1, p >= 0, n >= 0,
 * 0 <= q <= 16, damp finite and >= 0 (LX_ERR_INVALID_ARGUMENT); r + p <=
 * min(128, rows, cols, n'), rows * cols and n' * cols < 2^31
 * (LX_ERR_UNSUPPORTED); workspace 256-byte aligned,
 * lx_weighted_workspace_bytes(rows, cols, n, damp > 0, r, p) bytes (0 for
 * an unsupported shape). Asynchronous on `stream`; deterministic. */
size_t lx_weighted_workspace_bytes(int32_t rows, int32_t cols, int32_t n, int32_t damped, int32_t r, int32_t p);
lx_status lx_weighted_factors(const void* w_dom, const void* w_mem, lx_dtype dtype, int32_t rows, int32_t cols,
                              const int32_t* perm, int32_t perm_axis, const void* x, lx_dtype x_dtype, int32_t n,
                              double damp, int32_t r, int32_t p, int32_t q, const double* omega, float* A, float* B,
                              double* sigma, void* workspace, size_t workspace_bytes, void* stream);

/* Routing bucketing alone (the first step of every forward), exposing the
 * arrays of one tree level `level` (0 = anchors, n_levels = experts). It
 * organises the sharing of Sec. 5.1 ("Amortized forward pass"): the terms an
 * anchor or a tree node contributes are computed once per token that selects
 * any expert below it, so each level gets one row per distinct (token, node)
 * pair, and each slot the row it reads:
 *   row_token   [T * min(k, N_level)] (only the first node_offsets[N] entries
 *               are written): tokens of the unique (token, node) pairs, sorted
 *               by (node, token);
 *   node_offsets [N_level + 1]: exclusive prefix sum of rows per node;
 *   slot_row    [T * k]: row of the pair (t, node of slot t*k+j), or -1 for a
 *               dropped or invalid slot.
 * Deterministic: equal inputs give bit-identical arrays. Any of the three
 * output pointers may be NULL. Uses the forward's workspace size. */
lx_status lx_bucket(const lx_tree_layer* layer, int32_t T, int32_t k,
                    const int32_t* topk_ids, int32_t level, int32_t* row_token,
                    int32_t* node_offsets, int32_t* slot_row, void* workspace,
                    size_t workspace_bytes, void* stream);

/* Switch for the auxiliary stream of the forward entry points (see
 * "Auxiliary stream" above): enable = 1 lets prefill-sized forwards fork
 * their correction chains onto it, 0 (the default) keeps every launch on the
 * caller's stream. Process-wide; returns the previous setting. Results are
 * bitwise the same either way. No device call is made. */
int32_t lx_set_aux_stream(int32_t enable);

/* Device status bits (LX_DEVFLAG_*) of the last call that used `workspace`.
 * Synchronizes `stream`. */
lx_status lx_read_device_status(const void* workspace, void* stream, uint32_t* flags);

/* Optional kernel timing. While enabled, every kernel the library launches is
 * bracketed by HIP events recorded on the launch stream. lx_profile_collect
 * waits for the recorded events and adds their durations to per-kernel
 * totals; lx_profile_entry reads total i (name is a static string). Not
 * thread-safe; meant for benchmarks. */
lx_status lx_profile_enable(int32_t on);
lx_status lx_profile_collect(void);
int32_t lx_profile_count(void);
lx_status lx_profile_entry(int32_t i, const char** name, int64_t* launches, double* total_ms);
lx_status lx_profile_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* LOREX_H */
