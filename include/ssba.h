/*
 * ssba.h -- C ABI of the Shift Sparse Block Attention (SSBA) forward pass for
 * AMD Instinct MI355X (gfx950).
 *
 * SSBA (ElasticDiT, Section 2.2) is masked softmax attention over a diffusion
 * transformer's [text; image] token sequence.  The image tokens form an
 * H_g x W_g grid.  Per layer the grid origin is shifted by Delta (Section
 * 2.2.2, torch.roll semantics) and cut into Bt x Bt blocks.  Each image query
 * block keeps a subset of image key blocks (the gate).  Text tokens see
 * everything and are seen by everything (Algorithm 1, pad step).
 *
 * Gates (all four emit the same index layout, consumed by ssba_forward):
 *   SSBA_GATE_TOPK   -- Section 2.2.1 "Block Compression", "Affinity Matrix",
 *                       "Top-k Gating" (Eq. 1; Algorithm 1, pool/affinity/
 *                       top-k steps): per-block pooled Q and K, S = q_b k_b^T,
 *                       keep the `keep` largest entries of each row of S
 *                       (i.e. drop the floor(T_b * rho) smallest); ties keep
 *                       the lower key-block index; +0 == -0; NaN ranks last.
 *                       Pooled values are sums (mean x Bt^2), in fp64, added
 *                       in slot order; S is summed over channels in order,
 *                       without fused multiply-add.  Lists are therefore
 *                       bit-reproducible.
 *   SSBA_GATE_TOPK_SHARED -- the top-k gate with one score shared by all heads
 *                       of a batch element: S = sum over heads of the per-head
 *                       S_h (each as for TOPK), added in head order 0..H-1 in
 *                       fp64; every head receives the same kept lists.  The
 *                       paper states one gate per attention call over its
 *                       channels (Section 2.2.1); this is the shared variant.
 *   SSBA_GATE_WINDOW -- control gate: block i sees block j iff both lie in one
 *                       win_h x win_w window of blocks of the shifted frame.
 *   SSBA_GATE_DENSE  -- every block sees every block (zero sparsity).
 *
 * Sequence layout: T = n_text + grid_h * grid_w rows; text rows first; image
 * row n_text + y * grid_w + x holds grid token (y, x).  Q, K, V and O share one
 * element-stride triple (stride_b, stride_h, stride_t); the channel stride is 1.
 * Passing all three strides as 0 selects the contiguous [B, H, T, D] layout.
 * bf16 tensors must be 16-byte aligned with strides that are multiples of 8
 * elements (16-byte row loads); f32 tensors 4-byte aligned.
 *
 * Shifted frame: with (sy, sx) reduced mod (grid_h, grid_w), block t =
 * (ty, tx) (row-major over the n_y x n_x block grid) and slot s (row-major
 * inside the block) hold the image token at
 *   y = (ty * Bt + s / Bt - sy) mod grid_h,   x = (tx * Bt + s % Bt - sx) mod grid_w.
 * The shift is applied through this address map: no data is moved.
 *
 * Ownership and threading: the caller allocates and owns every buffer (device
 * memory, e.g. torch tensors).  The library allocates no device memory, keeps
 * no per-call state and may be called from several host threads.  Every call
 * is asynchronous on the caller's HIP stream (`hip_stream` = hipStream_t, NULL
 * for the null stream); only ssba_read_device_status synchronizes.
 *
 * Errors: descriptor and pointer checks happen before anything is launched;
 * on a non-zero status nothing has been enqueued and outputs are untouched.
 * SSBA_ERR_HIP reports a failed launch (hipGetLastError).
 *
 * Buffer sizes: every entry point that takes `index` or `scratch` has an
 * `_ex` form that also takes their sizes in bytes (`index_bytes`,
 * `scratch_bytes`) and returns SSBA_ERR_WORKSPACE, before anything is
 * launched, when a buffer is shorter than the call needs (the sizes that
 * ssba_workspace_size, ssba_layers_workspace_size or
 * ssba_backward_workspace_size report).  The forms without sizes check
 * nothing: the caller vouches for the buffers.
 */
#ifndef SSBA_H_
#define SSBA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSBA_ABI_VERSION 3

typedef enum {
  SSBA_OK = 0,
  SSBA_ERR_ARG = 1,          /* null pointer, bad enum, bad keep / window   */
  SSBA_ERR_SHAPE = 2,        /* non-positive sizes, grid not a multiple of Bt */
  SSBA_ERR_UNSUPPORTED = 3,  /* head_dim / tile / block count not built     */
  SSBA_ERR_WORKSPACE = 4,    /* index / scratch buffer shorter than needed  */
  SSBA_ERR_NONFINITE = 5,    /* gate saw a NaN/Inf affinity (device status) */
  SSBA_ERR_HIP = 6           /* HIP launch or copy failure                  */
} ssba_status;

typedef enum { SSBA_DT_BF16 = 0, SSBA_DT_F32 = 1 } ssba_dtype;
typedef enum {
  SSBA_GATE_TOPK = 0,
  SSBA_GATE_WINDOW = 1,
  SSBA_GATE_DENSE = 2,
  SSBA_GATE_TOPK_SHARED = 3
} ssba_gate;

typedef struct ssba_desc {
  int32_t batch, heads, head_dim;  /* B >= 1, H >= 1, D in {64, 128}               */
  int32_t grid_h, grid_w, tile;    /* Bt in {4, 8, 16}; grid_h, grid_w multiples of Bt */
  int32_t shift_y, shift_x;        /* Delta, any sign, reduced mod the grid          */
  int32_t n_text;                  /* >= 0 text tokens, stored before the image rows */
  int32_t gate;                    /* ssba_gate                                      */
  int32_t keep;                    /* TOPK, TOPK_SHARED: kept key blocks per query block, 1..T_b */
  int32_t win_h, win_w;            /* WINDOW: window in blocks; n_y % win_h == n_x % win_w == 0 */
  int32_t dtype;                   /* ssba_dtype of Q, K, V and O                    */
  float softmax_scale;             /* <= 0 selects 1 / sqrt(head_dim)                */
  int64_t stride_b, stride_h, stride_t; /* element strides; all 0 = contiguous     */
} ssba_desc;

/* Returns SSBA_ABI_VERSION. */
int ssba_abi_version(void);

/* Static, never-NULL description of a status code. */
const char* ssba_status_str(ssba_status s);

/* Device bytes the caller must provide.
 *   index_bytes   = 4 * B * H * T_b * (1 + T_b): the index of ssba_build_index.
 *   scratch_bytes = TOPK: 16 * B * H * T_b * D (fp64 pooled q_b and k_b)
 *                   + 4 * B * H * T_b (per-row status flags);
 *                   TOPK_SHARED: as TOPK + 8 * B * H * T_b^2 (fp64 per-head
 *                   affinity rows);
 *                   WINDOW / DENSE: 4 * B * H * T_b.
 * Either output pointer may be NULL.  T_b = grid_h * grid_w / Bt^2. */
ssba_status ssba_workspace_size(const ssba_desc* d, size_t* index_bytes, size_t* scratch_bytes);

/* Gate (Section 2.2.1 Block Compression / Affinity / Top-k Gating; Algorithm 1
 * pool, affinity, top-k and expand steps).  Writes `index`, int32
 * [B][H][T_b][1 + T_b]: entry 0 = count of kept key blocks, then their block
 * ids ascending, then -1 padding.  TOPK and TOPK_SHARED read the image rows of
 * q and k (dtype d->dtype, layout above); WINDOW and DENSE read neither (q, k
 * may be NULL).
 * `scratch` (scratch_bytes, 16-byte aligned) is overwritten; its status
 * flags are read by ssba_read_device_status. */
ssba_status ssba_build_index(const ssba_desc* d, const void* q, const void* k,
                             int32_t* index, void* scratch, void* hip_stream);

/* ssba_build_index with the sizes of `index` and `scratch` in bytes. */
ssba_status ssba_build_index_ex(const ssba_desc* d, const void* q, const void* k, int32_t* index,
                                size_t index_bytes, void* scratch, size_t scratch_bytes, void* hip_stream);

/* SSBA attention (Algorithm 1, attend step): O = softmax(scale * Q K^T + mask) V
 * where an image query in block i sees the image keys of the blocks listed in
 * index[b][h][i] and every text key; a text query sees every key.  Masked
 * blocks are never loaded.  Writes all T rows of o (text rows included);
 * the image rows are the layer output of Algorithm 1's return step.
 * bf16: products and accumulation in fp32 (MFMA), probabilities rounded to
 * bf16 before the value product, output rounded to bf16.  f32: fp32 throughout.
 * `index` must come from ssba_build_index with the same grid/tile/shift, or
 * hold lists of the same layout (counts in 0..T_b, ids in 0..T_b-1; other
 * contents are undefined behaviour).  A query that sees no key (an empty
 * list and no text tokens) gets a row of zeros. */
ssba_status ssba_forward(const ssba_desc* d, const void* q, const void* k, const void* v,
                         const int32_t* index, void* o, void* hip_stream);

/* ssba_forward with the size of `index` in bytes. */
ssba_status ssba_forward_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                            const int32_t* index, size_t index_bytes, void* o, void* hip_stream);

/* Dense attention in the same kernel family (the zero-sparsity control of
 * Section 2.2.1's cost comparison): every query sees all T keys; the gate,
 * shift and index are ignored. */
ssba_status ssba_forward_dense(const ssba_desc* d, const void* q, const void* k, const void* v,
                               void* o, void* hip_stream);

/* Gate and attention in one call (the top-k gate fused into the attention
 * kernel, Section 2.2.1 and Algorithm 1 pool through attend steps): the same
 * results as ssba_build_index followed by ssba_forward -- `index` receives
 * bit-identical index rows, `scratch` the same status flags, `o` the same
 * output -- with one launch fewer.  d->gate must be SSBA_GATE_TOPK or
 * SSBA_GATE_TOPK_SHARED.  For TOPK with bf16 inputs, 8x8 blocks, head_dim 64
 * or 128 and at most 64 blocks it launches the pooling kernel and an
 * attention kernel in which each query block forms its affinity row from the
 * pooled sums and ranks it before attending; other shapes and the shared
 * gate run the two calls.  Buffers, sizes and alignment as for
 * ssba_build_index and ssba_forward. */
ssba_status ssba_forward_topk(const ssba_desc* d, const void* q, const void* k, const void* v,
                              int32_t* index, void* scratch, void* o, void* hip_stream);

/* The two launches of ssba_forward_topk's fused form, callable one at a time
 * (Algorithm 1: ssba_pool_keys_ex is the pooling of K, Eq. 1;
 * ssba_forward_gated_ex the affinity, ranking and attention steps).
 * ssba_forward_topk_ex with the fused form is exactly ssba_pool_keys_ex then
 * ssba_forward_gated_ex on one stream.  Both need d->gate == SSBA_GATE_TOPK,
 * bf16, 8x8 blocks, head_dim 64 or 128 and at most 64 blocks, and return
 * SSBA_ERR_UNSUPPORTED otherwise (ssba_forward_topk then runs the two calls).
 * ssba_pool_keys_ex writes the pooled key sums of every (batch, head) into
 * `scratch` (fp64, at the place the gated launch reads them); it reads only k.
 * ssba_forward_gated_ex reads those sums, so `scratch` must hold what
 * ssba_pool_keys_ex wrote for the same k and descriptor (anything else gives
 * undefined index rows, never an out-of-bounds access: every id is range-
 * checked); it writes index, the status flags in scratch and o, as
 * ssba_forward_topk does.  Sizes, alignment and errors as for
 * ssba_forward_topk_ex. */
ssba_status ssba_pool_keys_ex(const ssba_desc* d, const void* k, void* scratch, size_t scratch_bytes,
                              void* hip_stream);
ssba_status ssba_forward_gated_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                  int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                  void* o, void* hip_stream);

/* ssba_forward_topk with the sizes of `index` and `scratch` in bytes. */
ssba_status ssba_forward_topk_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                 int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                 void* o, void* hip_stream);

/* Training forward: ssba_forward plus `lse`, fp32 [B][H][T], the natural-log
 * log-sum-exp of each row's scaled scores (log of the softmax normaliser,
 * log sum_j exp(scale q . k_j) over the row's visible keys), which
 * ssba_backward needs.  bf16, head_dim 64 or 128, 8x8 or 16x16 blocks (the
 * MFMA kernel); other shapes return SSBA_ERR_UNSUPPORTED.  `lse` 4-byte
 * aligned, caller-owned. */
ssba_status ssba_forward_train(const ssba_desc* d, const void* q, const void* k, const void* v,
                               const int32_t* index, void* o, float* lse, void* hip_stream);

/* ssba_forward_train with the size of `index` in bytes. */
ssba_status ssba_forward_train_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                  const int32_t* index, size_t index_bytes, void* o, float* lse,
                                  void* hip_stream);

/* Device bytes of the scratch ssba_backward needs (256-byte aligned buffer):
 * fp32 [B][H][T] twice (the log-sum-exp in log2 units and rowsum(dO * O)), a
 * 64-bit mask of kept blocks per query block, [B][H][T_b], and the order in
 * which the key-side kernel takes the key blocks, int32 [B][H][T_b]; each
 * region rounded up to 256 bytes. */
ssba_status ssba_backward_workspace_size(const ssba_desc* d, size_t* scratch_bytes);

/* Backward of the SSBA attention with the gate held fixed (the kept lists
 * carry no gradient): given Q, K, V, the forward output O and its lse (from
 * ssba_forward_train with the same descriptor and index) and the upstream
 * gradient dout (dO), writes
 *   dq = scale dS K,  dk = scale dS^T Q,  dv = P^T dO,
 * with P = softmax(scale Q K^T + mask) recomputed from lse, dP = dO V^T and
 * dS = P * (dP - rowsum(dO * O)).  The mask is that of ssba_forward: image
 * queries see their kept blocks and the text keys, text queries see every
 * key.  All tensors bf16 with the descriptor's layout (dq, dk, dv written in
 * full, every row); products on MFMA with fp32 accumulation, P and dS rounded
 * to bf16 before their products.  bf16, 8x8 or 16x16 blocks, head_dim 64 or
 * 128, at most 64 blocks; other shapes return SSBA_ERR_UNSUPPORTED.  The gate fields
 * of the descriptor are not used. */
ssba_status ssba_backward(const ssba_desc* d, const void* q, const void* k, const void* v, const void* o,
                          const void* dout, const float* lse, const int32_t* index, void* dq, void* dk,
                          void* dv, void* scratch, void* hip_stream);

/* ssba_backward with the sizes of `index` and `scratch` in bytes. */
ssba_status ssba_backward_ex(const ssba_desc* d, const void* q, const void* k, const void* v, const void* o,
                             const void* dout, const float* lse, const int32_t* index, size_t index_bytes,
                             void* dq, void* dk, void* dv, void* scratch, size_t scratch_bytes,
                             void* hip_stream);

/* The rotary step of Algorithm 1 fused into the pooling pre-pass (bf16, 8x8
 * blocks, D 64 or 128, at most 64 blocks; else SSBA_ERR_UNSUPPORTED): writes
 * the rotated Q and K to q_rope and k_rope (layout of the descriptor; text
 * rows copied unchanged) and the pooled sums of the rotated keys to scratch,
 * as ssba_pool_keys_ex does for k.  The rotation (the paper names the step,
 * not its variant) is the 2-D axial one: channels [0, D/2) turn with the
 * token's row in the image grid, [D/2, D) with its column; pair i of a half
 * (channels 2i, 2i+1) by the angle pos * theta^(-i / (D/4)), computed in
 * fp64 and rounded to bf16 (nearest even).  theta <= 0 selects 10000; a
 * non-finite theta is SSBA_ERR_ARG.  q_rope and k_rope may be q and k (in
 * place) and must not otherwise overlap an input.  Sizes and errors as
 * ssba_pool_keys_ex. */
ssba_status ssba_rope_pool_keys_ex(const ssba_desc* d, const void* q, const void* k, void* q_rope, void* k_rope,
                                  float theta, void* scratch, size_t scratch_bytes, void* hip_stream);

/* ssba_forward_topk with the rotary step first (Algorithm 1 in full): the
 * pre-pass above, then the gated attention on the rotated Q and K.  Writes
 * q_rope, k_rope, the index and O; the results equal ssba_forward_topk on
 * q_rope and k_rope.  Shapes, sizes and errors as ssba_forward_gated_ex. */
ssba_status ssba_forward_topk_rope_ex(const ssba_desc* d, const void* q, const void* k, const void* v,
                                     void* q_rope, void* k_rope, float theta, int32_t* index, size_t index_bytes,
                                     void* scratch, size_t scratch_bytes, void* o, void* hip_stream);

/* Largest scratch (bytes) that ssba_forward_topk_noalloc provides: the
 * fixed device array it uses in place of a caller buffer. */
#define SSBA_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): the same call
 * and results as ssba_forward_topk, with the scratch taken from a fixed array
 * of SSBA_NOALLOC_SCRATCH_BYTES in device memory that the library holds on
 * every device it runs on until the process ends.  The caller still passes
 * the inputs and the outputs (`index`, `index_bytes`, `o`).  Returns
 * SSBA_ERR_WORKSPACE, before anything is launched, when the scratch that
 * ssba_workspace_size reports for `d` exceeds SSBA_NOALLOC_SCRATCH_BYTES, or
 * when `index_bytes` is short.  Allocates nothing.  Every call on one device
 * shares that device's array: calls that overlap on a device (several
 * streams or threads) race; calls ordered on one stream do not.  The status
 * flags of the gate stay in the array, so ssba_read_device_status has no
 * buffer to read for this call. */
ssba_status ssba_forward_topk_noalloc(const ssba_desc* d, const void* q, const void* k, const void* v,
                                      int32_t* index, size_t index_bytes, void* o, void* hip_stream);

/* One layer of a stack run by ssba_forward_layers. */
typedef struct ssba_layer {
  const void* q;    /* this layer's Q, K, V and output O (layout of the descriptor) */
  const void* k;
  const void* v;
  void* o;
  int32_t keep;     /* top-k gates: kept key blocks per query block, 1..T_b      */
  int32_t skip;     /* nonzero: the layer is skipped (nothing runs, o untouched)  */
} ssba_layer;

/* Device bytes ssba_forward_layers needs for n_layers layers of descriptor d
 * (d->keep is not used): index_bytes = n_layers * the index of one call;
 * scratch_bytes = n_layers * the scratch of one call rounded up to 256 bytes.
 * Layer l's slices start at l * (index_bytes / n_layers) and
 * l * (scratch_bytes / n_layers). */
ssba_status ssba_layers_workspace_size(const ssba_desc* d, int n_layers, size_t* index_bytes,
                                       size_t* scratch_bytes);

/* A stack of SSBA layer calls on one stream (Section 2.2.2 offset alternation;
 * the per-layer sparsity of the layer-importance-aware scheme, Table 2; the
 * skipped blocks of Sparse-Depth Pruning, Section 2.1.2).  Layer l uses the
 * offset (d->shift_y, d->shift_x) on even l and its negation on odd l (the
 * paper's rule with (Bt/2, Bt/2)), layers[l].keep for the top-k gates, and
 * does nothing if layers[l].skip.  Each layer's results equal one
 * ssba_forward_topk call (top-k gates) or ssba_build_index + ssba_forward
 * (static gates) with that layer's descriptor, index slice and scratch slice.
 * Static gates depend only on the frame, so the index is built once per
 * offset parity (in the slice of the first layer of that parity that runs)
 * and reused by the later layers of that parity, whose slices are left
 * untouched.  Where the attention runs on the matrix-core kernels (bf16,
 * D 64/128, 8x8 or 16x16 blocks, T_b <= 64), up to 32 running layers share
 * each launch: for the top-k gate one launch pools their keys and one runs
 * their gated attention; for the head-shared gate one launch per gate step
 * builds their indices; then (for it and the static gates) one launch runs
 * their attention.  Each workgroup computes what it computes in a one-layer
 * launch, so the results are the same bits as one call per layer.  Every
 * layer is checked before anything is launched; a HIP launch failure stops
 * the stack after the layers already enqueued. */
ssba_status ssba_forward_layers(const ssba_desc* d, const ssba_layer* layers, int n_layers,
                                int32_t* index, void* scratch, void* hip_stream);

/* ssba_forward_layers with the sizes of `index` and `scratch` in bytes (the
 * whole stack's, as ssba_layers_workspace_size reports them). */
ssba_status ssba_forward_layers_ex(const ssba_desc* d, const ssba_layer* layers, int n_layers,
                                   int32_t* index, size_t index_bytes, void* scratch, size_t scratch_bytes,
                                   void* hip_stream);

/* Name of the attention kernel that ssba_forward (mode 0), ssba_forward_dense
 * (mode 1) or ssba_forward_topk (mode 2) launches for this descriptor, as
 * profilers show it without namespace and arguments (e.g.
 * "k_attn_mfma<64, 3, false, false>"); NULL if the descriptor or mode is
 * invalid.  Static storage; launches nothing. */
const char* ssba_forward_kernel(const ssba_desc* d, int mode);

/* Synchronizes `hip_stream`, then reads the status flags that the last
 * ssba_build_index left in `scratch` (same descriptor): SSBA_OK, or
 * SSBA_ERR_NONFINITE if any affinity row held a NaN or Inf (top-k gates only;
 * for the shared gate, the summed row).  d->keep is not used here. */
ssba_status ssba_read_device_status(const ssba_desc* d, const void* scratch, ssba_status* out,
                                    void* hip_stream);

/* ssba_read_device_status with the size of `scratch` in bytes. */
ssba_status ssba_read_device_status_ex(const ssba_desc* d, const void* scratch, size_t scratch_bytes,
                                       ssba_status* out, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* SSBA_H_ */
