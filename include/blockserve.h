/*
 * blockserve.h -- C ABI of the MI355X (gfx950) mixed-state denoising step.
 *
 * One step of BlockServe's block-grained continuous batching (Zhu et al.,
 * "BlockServe: Block-Grained Continuous Batching for High-Throughput Diffusion
 * LLM Serving"): every request of a heterogeneous batch sits at its own block
 * index; the step gathers each request's active block, attends it against the
 * request's dual KV cache, decodes it with confidence-threshold parallel
 * decoding, and scatters the result back. At block boundaries the dense KV box
 * is rewritten when requests are evicted and admitted.
 *
 * Conventions shared by every call
 * --------------------------------
 * Request descriptor (Section "Problem formulation"): a request has prompt
 * length p, generation length g, block length L and current block index k
 * (the paper's b_i), 0 <= k < K = ceil(g / L). Block k covers logical
 * positions [s, s + B) with s = p + k L and B = min(L, g - k L); the request's
 * logical row [0, p + g) holds prompt, generated blocks and the still-masked
 * suffix. Logical position t lives at column off + t of row `row` of every
 * dense [R][W] tensor (paragraph "Logical positional alignment": left padding,
 * position ids counted from the first non-padding cell).
 * A descriptor array is valid when L >= 1 and, for each entry, p >= 0, g >= 1,
 * 0 <= k < K, 0 <= row < R, off >= 0, off + p + g <= W, and no two entries
 * share a row.
 *
 * Memory: every tensor argument is a DEVICE pointer owned by the caller (this
 * library allocates no tensor memory). Descriptor and segment arrays are HOST
 * pointers, read during the call only. Tensors are dense, row-major, in the
 * layouts stated per call; bf16 is the IEEE upper half of fp32, stored as
 * 16-bit words.
 *
 * Streams: `stream` is a hipStream_t (NULL = the legacy default stream). Every
 * call only enqueues work on it; results are valid after the stream (or an
 * event recorded on it) has completed, and device pointers must stay valid
 * until then. A call does not wait for the device, with one bounded
 * exception: a context keeps the device copies of its descriptor sets in
 * upload slots and adds a slot rather than overwrite one that queued work
 * still reads; only when 256 distinct descriptor sets of one context are in
 * flight at once does a call wait for the oldest of them to be read.
 *
 * Errors: every int-returning call returns a bs_status. Arguments are checked
 * on the host BEFORE anything is enqueued, so a failing call launches nothing
 * and leaves every tensor untouched; bs_last_error() gives the detail.
 *
 * Threads: a bs_ctx holds the descriptor upload slots; use one context per
 * host thread. Calls on one context may target different streams.
 */
#ifndef BLOCKSERVE_H
#define BLOCKSERVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bs_req_desc {
  int32_t p;    /* prompt length p_i */
  int32_t g;    /* generation length g_i */
  int32_t k;    /* current block index (b_i), 0 <= k < ceil(g / L) */
  int32_t row;  /* row of the dense box holding this request */
  int32_t off;  /* column of logical position 0 in that row */
} bs_req_desc;

typedef struct bs_copy_seg {
  int32_t src_kind; /* 0: old cache box, 1: staging box */
  int32_t src_row;
  int32_t src_col;
  int32_t dst_row;
  int32_t dst_col;
  int32_t len;      /* cached positions to copy (>= 0) */
} bs_copy_seg;

typedef enum bs_dtype { BS_F32 = 0, BS_BF16 = 1 } bs_dtype;

typedef enum bs_status {
  BS_OK = 0,
  BS_ERR_INVALID_ARG = 1,  /* null pointer, bad enum, negative size, bad stride */
  BS_ERR_UNSUPPORTED = 2,  /* shape/dtype combination the library does not serve */
  BS_ERR_DESCRIPTOR = 3,   /* descriptor array invalid (see conventions above) */
  BS_ERR_OVERLAP = 4,      /* copy destinations intersect, or a source aliases a destination */
  BS_ERR_WORKSPACE = 5,    /* workspace missing or smaller than the size query returns */
  BS_ERR_HIP = 6           /* HIP runtime or launch failure */
} bs_status;

typedef struct bs_ctx bs_ctx;

/* Create a context bound to HIP device `device` (it becomes current while the
 * library works). The context owns only pinned host staging memory and device
 * upload slots for descriptors and work lists (allocated as calls need them),
 * plus four 512 KiB pinned stages for bs_mixed_state_step_noalloc, allocated
 * here; it also resolves the device address of the library's static array
 * for that call. *out is NULL on failure. */
int bs_create(bs_ctx** out, int device);

/* Wait for every upload slot to drain, then free the context (NULL is OK). */
int bs_destroy(bs_ctx* ctx);

/* Static text for a status code. */
const char* bs_status_string(int status);

/* Detail of the last failure on this context ("" if none; ctx may be NULL,
 * which returns the detail of the last failure of a context-free call). */
const char* bs_last_error(const bs_ctx* ctx);

/* Host-only check of a descriptor array against block length L and an
 * R x W box (the rules under "Conventions"). Touches no device. */
int bs_validate_requests(const bs_req_desc* reqs, int n, int L, int R, int W);

/* Host-only check of a K4 segment array (the rules of bs_kv_scatter_compact
 * below): every segment inside its boxes (source: R_src x W_src for src_kind
 * 0, R_stg x W_stg for src_kind 1; destination R_dst x W_dst), destination
 * ranges pairwise disjoint, and, when src_is_dst (stg_is_dst) is nonzero, no
 * source range of that kind meeting any destination range. Segments of length
 * 0 copy nothing and never overlap. Returns BS_OK, BS_ERR_INVALID_ARG or
 * BS_ERR_OVERLAP (detail in bs_last_error(NULL)). Touches no device. */
int bs_validate_segments(const bs_copy_seg* segs, int nseg, int R_src, int W_src, int R_stg, int W_stg, int R_dst,
                         int W_dst, int src_is_dst, int stg_is_dst);

/*
 * K1 -- gather of the active blocks (paragraph "Vectorized mixed-schedule
 * execution": gather extracts each request's active block region into a
 * compact tensor).
 *   dst[i][j] = src[row_i][off_i + s_i + j]   for j < B_i, else all-zero bytes
 *   pos_out[i][j] = s_i + j                   for j < B_i, else -1
 * src: dense [R][W] elements of `elem_bytes` bytes (1, 2, 4, 8 or 16), rows
 * `src_row_stride_bytes` apart (>= W * elem_bytes). dst: compact [n][L]
 * elements, contiguous. pos_out: [n][L] int32 or NULL. n == 0 is a no-op.
 */
int bs_gather_active_blocks(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W,
                            const void* src, int64_t src_row_stride_bytes, int elem_bytes,
                            void* dst, int32_t* pos_out, void* stream);

/* Inverse of K1 (paragraph "Vectorized mixed-schedule execution": scatter
 * writes results back to the corresponding positions):
 *   dst[row_i][off_i + s_i + j] = src[i][j]   for j < B_i.
 * No other cell of dst is written. */
int bs_scatter_active_blocks(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W,
                             const void* src_compact, int elem_bytes, void* dst_dense,
                             int64_t dst_row_stride_bytes, void* stream);

/* K1 over several same-geometry tensors in one launch (the step gathers token
 * ids and mask bits together). Tensor k (0 <= k < ntensors <= 4) has its own
 * element size elem_bytes[k], dense row stride *_row_stride_bytes[k], dense
 * pointer and compact pointer; each is moved exactly as by the single-tensor
 * call above. The four arrays are host arrays of ntensors entries, read
 * before the call returns. pos_out as above (gather only). */
int bs_gather_active_blocks_n(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W, int ntensors,
                              const void* const* src, const int64_t* src_row_stride_bytes,
                              const int* elem_bytes, void* const* dst, int32_t* pos_out, void* stream);
int bs_scatter_active_blocks_n(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W, int ntensors,
                               const void* const* src_compact, const int* elem_bytes, void* const* dst_dense,
                               const int64_t* dst_row_stride_bytes, void* stream);

/*
 * K2 -- dual-cache block attention for one layer (paragraph "Vectorized
 * mixed-schedule execution": the active block is computed against the cached
 * KV and the fresh block KV is written in place at the physical offsets of the
 * request's current block only; dual cache = cached prefix + cached masked
 * suffix, the Fast-dLLM mechanism the paper integrates, Sections
 * "Experimental setup" and "Diffusion LLM Inference Optimization").
 * For request i, query head h (KV head c = h / (Hq / Hkv)) and block row
 * j < B_i, with keys/values = [cache cols off+[0,s) | k_new/v_new rows [0,B) |
 * cache cols off+[s+B, p+g)] of row_i, head c:
 *   out[i][j][h] = softmax(scale * q[i][j][h] . keys^T) . values
 * (bidirectional, no cross-request or padding keys). out rows j >= B_i are
 * written as zeros. scale <= 0 selects 1/sqrt(D).
 * Layouts (element type `dt` for all five tensors):
 *   q, out        [n][L][Hq][D]      k_new, v_new  [n][L][Hkv][D]
 *   k_cache, v_cache [R][Hkv][W][D]
 * write_back != 0 additionally stores k_new/v_new rows j < B_i into the cache
 * cells [off_i + s_i + j] of head c (no other cache cell is written); with 0
 * the caches are only read.
 * Prefix-cache layout (keys = prompt, decoded blocks and the active block,
 * without the masked suffix): pass g_i' = min(g_i, (k_i + 1) L) with the same
 * off_i; the cells past the active block are then never read.
 * Supported: Hq % Hkv == 0; BS_F32 with D % 4 == 0, D <= 256; BS_BF16 with
 * D in {64, 128}, L <= 64 and Hq / Hkv <= 8. All pointers
 * 16-byte aligned. Cache cells outside each request's logical row and the
 * stale block slot are never read (they may hold NaN).
 * ws: NULL, or a device workspace of ws_bytes bytes (contents on entry
 * ignored). Straggler handling (split-KV; the paper's straggler effect,
 * Introduction and RQ2): the BS_BF16 kernels hold a fixed number of rows at
 * once (one workgroup of G * ceil(L / 32) waves per CU, or four single-wave
 * rows per CU for MHA with L <= 32), so a batch of whole rows lasts at least
 * as long as its longest row. bs_attention_workspace_bytes(...) returns the
 * bytes of partial slots for a plan that cuts the longest rows into pieces of
 * 64-key tiles (each piece writes its un-normalised output, running max and
 * row sum; a merge launch combines them by log-sum-exp weights), or 0 when no
 * cut pays off (rows that already fill the GPU evenly, BS_F32, invalid
 * arguments). With
 * ws_bytes at least that size the call runs the plan, otherwise every row
 * whole; both agree within rounding (bf16 output). The plan depends only on
 * the arguments of the size query. Calls that may overlap (different
 * streams) need different workspaces.
 */
size_t bs_attention_workspace_bytes(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D,
                                    bs_dtype dt);
/*
 * Host only (no device work): the BS_BF16 attention's work list for these
 * arguments, in launch order, as 6 int32 per workgroup: request, KV head,
 * first 32-row block, first and one-past-last 64-key tile, partial slot (-1
 * for a whole row). split = 0 gives the whole-row list, 1 the split-KV plan
 * (the one bs_attention_workspace_bytes sizes). Writes min(*n_items,
 * max_items) entries to `items` (caller-owned), the list length to *n_items
 * and the plan's partial-slot count to *n_parts. BS_ERR_UNSUPPORTED outside
 * the bf16 kernels' shapes; descriptors are not validated.
 */
int bs_attention_work_list(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D, bs_dtype dt, int split,
                           int32_t* items, int max_items, int* n_items, int* n_parts);
int bs_dual_cache_block_attention(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int Hq,
                                  int Hkv, int D, bs_dtype dt, float scale, const void* q,
                                  const void* k_new, const void* v_new, void* k_cache,
                                  void* v_cache, int R, int W, int write_back, void* out,
                                  void* ws, size_t ws_bytes, void* stream);

/*
 * K3 -- confidence-aware parallel decode of the active blocks (paragraph
 * "Vectorized mixed-schedule execution": per-step transfer quota; greedy
 * decoding, "Implementation details"; Fast-dLLM's threshold rule integrated
 * unchanged). For request i let M = { j < B_i : masked[i][j] != 0 }. For j in M:
 *   x_j = argmax_v logits[i][j][v]                (ties: smallest v)
 *   c_j = 1 / sum_v exp(logits[i][j][v] - max_v)  (max softmax probability)
 * n_i = min(|M|, max(q_min, #{j in M : c_j >= tau})); the n_i most confident
 * positions of M (ties: smallest j) get tokens[i][j] = x_j, masked[i][j] = 0.
 * Every other cell of tokens/masked is left unchanged (no re-masking).
 * Outputs: n_unmasked[i] = n_i; done[i] = (n_i == |M|); eos_seen[i] = some
 * j < B_i has masked == 0 and tokens == eos_id after the update (always 0 when
 * eos_id < 0); conf_out[i][j] = c_j for j in M, -1 otherwise (conf_out may be
 * NULL). A request with M empty is a no-op with done = 1.
 * logits: [n][L] rows of V elements of `logits_dt`, row (i, j) starting at
 * logits + (i * L + j) * logits_row_stride elements (stride >= V, stride *
 * element size a multiple of 16 bytes, base 16-byte aligned). Only rows
 * j in M are read; their entries are finite or -inf (a vocabulary entry that
 * is ruled out), with at least one finite entry per row; NaN and +inf are
 * outside the contract. tokens [n][L] int32 and masked [n][L]
 * uint8 are updated in place. q_min >= 1 (at least one unmask per step while
 * any position is masked); L <= 64.
 * ws: device workspace of at least bs_decode_workspace_bytes(...) bytes,
 * 16-byte aligned; its contents on entry are ignored (it carries per-row
 * partial results between the call's two launches, and in the fused step
 * each request's block mask bits from its attention to its decode). Calls
 * that may overlap (different streams) need different workspaces.
 */
size_t bs_decode_workspace_bytes(int n, int L, int V, bs_dtype logits_dt);
int bs_parallel_decode(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int V,
                       bs_dtype logits_dt, const void* logits, int64_t logits_row_stride,
                       int32_t* tokens, uint8_t* masked, float tau, int32_t q_min, int32_t eos_id,
                       int32_t* n_unmasked, uint8_t* done, uint8_t* eos_seen, float* conf_out,
                       void* ws, size_t ws_bytes, void* stream);

/*
 * K3 with the output head fused in (paragraph "Vectorized mixed-schedule
 * execution"; greedy parallel decoding, "Implementation details"): the same
 * decoding step as bs_parallel_decode, with the logits of each masked
 * position produced from its final hidden state,
 *   logits[i][j][v] = sum_k hidden[i][j][k] * w_vocab[v][k],
 * accumulated in fp32 and reduced on the fly (they never reach memory).
 * Only rows j < B_i with masked[i][j] != 0 are projected; other hidden rows
 * are never read (they may hold NaN).
 * The output-head matrix is passed in the packed layout bs_lm_head_pack
 * writes (once per model): contiguous 16 KiB slabs that the kernel's LDS
 * stages copy whole.
 * hidden: [n][L][d] bf16, 16-byte aligned. w_packed: bs_lm_head_pack's output
 * for the same V and d. dt must be BS_BF16; d a multiple of 32; L <= 64;
 * q_min >= 1. tokens, masked, tau, q_min, eos_id and the outputs are as in
 * bs_parallel_decode (compact [n][L] block state, updated in place).
 * ws: device workspace of at least bs_lm_head_workspace_bytes(n, L, V)
 * bytes, 16-byte aligned; contents on entry are ignored (it carries the row
 * list and partial results between the call's launches). Calls that may
 * overlap need different workspaces.
 */
size_t bs_lm_head_workspace_bytes(int n, int L, int V);
int bs_lm_head_decode(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int d, int V, bs_dtype dt,
                      const void* hidden, const void* w_packed, int32_t* tokens, uint8_t* masked, float tau,
                      int32_t q_min, int32_t eos_id, int32_t* n_unmasked, uint8_t* done, uint8_t* eos_seen,
                      float* conf_out, void* ws, size_t ws_bytes, void* stream);

/*
 * Re-layout of the output-head matrix for bs_lm_head_decode (done once, when
 * the model is loaded). w_vocab: [V] rows of w_row_stride bf16 elements
 * (stride >= d, a multiple of 8), 16-byte aligned, read only. w_packed:
 * device buffer of at least bs_lm_head_pack_bytes(V, d) bytes, 16-byte
 * aligned, fully written: for each 256-row vocabulary tile t and 32-wide K
 * slice s, a 16 KiB slab at element offset (t * (d / 32) + s) * 8192 holds
 * rows 256 t .. 256 t + 255 (zero past V) as 64-byte rows whose 16-byte chunk
 * c sits in slot c ^ ((row >> 2) & 3). dt must be BS_BF16, d a multiple of 32.
 */
size_t bs_lm_head_pack_bytes(int V, int d);
int bs_lm_head_pack(bs_ctx* ctx, const void* w_vocab, int64_t w_row_stride, int V, int d, bs_dtype dt,
                    void* w_packed, size_t packed_bytes, void* stream);

/*
 * Dual-cache refresh of one layer at a block start, and the prefill of newly
 * admitted rows (the dual cache of Fast-dLLM that the paper integrates:
 * cached prefix and masked-suffix KV are recomputed by a forward over the
 * whole row when a block starts, Sections "Experimental setup" and "Diffusion
 * LLM Inference Optimization"; paragraph "Logical positional alignment":
 * position ids count the real tokens of the left-padded row, so rotary
 * embeddings see each request's own distances).
 * For request i (row r, offset off, logical length len = p + g), cell
 * t < len and position id t (the cumulative count over the row's attention
 * mask, minus one):
 *   K_t = rope(k[r][off + t], t),  Q_t = rope(q[r][off + t], t)
 *   k_cache[r][c][off + t] = K_t,c,  v_cache[r][c][off + t] = v[r][off + t][c]
 *   out[r][off + t][h] = softmax(scale * Q_t,h . K_c^T) V_c over keys t' < len
 * (bidirectional; query head h reads KV head c = h / (Hq / Hkv)).
 * rope(x, t) turns feature pair (f, f + D/2), f < D/2, by the angle
 * t * rope_base^(-2 f / D) (RoFormer; the rotate-half pairing); rope_base
 * <= 0 disables the rotation. scale <= 0 selects 1/sqrt(D).
 * Layouts (bf16): q, out [R][W][Hq][D] and k, v [R][W][Hkv][D] (token-major
 * projections of the dense box); k_cache, v_cache [R][Hkv][W][D]. Only the
 * requests' logical cells are read (padding may hold NaN) or written (every
 * other cell of out and the caches is left unchanged). q, k, v must not
 * overlap the caches or out. The descriptors are validated as everywhere
 * (L and k only there); R * W * Hq < 2^31; n <= 65535.
 * Supported: dt = BS_BF16, D = 128, Hq % Hkv == 0. All pointers 16-byte
 * aligned. Two launches on `stream` (keys and values, then attention).
 */
int bs_dual_cache_refresh(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D,
                          bs_dtype dt, float scale, float rope_base, const void* q, const void* k,
                          const void* v, int R, int W, void* k_cache, void* v_cache, void* out,
                          void* stream);

/*
 * K4 -- KV scatter/compaction at a block boundary (Algorithm 1: completed
 * requests leave and new ones are admitted at the block boundary; Eq. 1
 * discussion: the box shrinks without explicit reclamation; paragraph
 * "Vectorized mixed-schedule execution": the frozen prefix cache survives
 * batch reconfiguration). For every segment, layer l < n_layers, KV head
 * h < Hkv and t < len, for K and for V:
 *   dst[l][dst_row][h][dst_col + t] = S[l][src_row][h][src_col + t]
 * where S is the old box (src_kind 0) or the staging box (src_kind 1).
 * Boxes are [n_layers][R_x][Hkv][W_x][D] of `dt`, layers `*_layer_stride`
 * BYTES apart (>= R_x * Hkv * W_x * D * elem). Every other dst cell is left
 * unchanged. Rules (BS_ERR_OVERLAP otherwise): destination ranges are
 * pairwise disjoint; when a source box is the destination box (same
 * pointers), no source range of a segment intersects any destination range.
 * A segment of length 0 copies nothing and takes no part in these rules
 * (bs_validate_segments applies the same checks on the host alone).
 * D * elem must be a multiple of 16 bytes. stg_* may be NULL when no segment
 * has src_kind 1; src_* may be NULL when none has src_kind 0.
 */
int bs_kv_scatter_compact(bs_ctx* ctx, const bs_copy_seg* segs, int nseg, int n_layers, int Hkv,
                          int D, bs_dtype dt, const void* src_k, const void* src_v,
                          int64_t src_layer_stride, int R_src, int W_src, const void* stg_k,
                          const void* stg_v, int64_t stg_layer_stride, int R_stg, int W_stg,
                          void* dst_k, void* dst_v, int64_t dst_layer_stride, int R_dst, int W_dst,
                          void* stream);

/*
 * One mixed-state denoising step in one call (Algorithm 1's inner loop body;
 * paragraph "Vectorized mixed-schedule execution": every request advances its
 * own active block in the same batched step). Enqueues, in order: K2 for each
 * layer l < n_layers on that layer's tensors (q[l], k_new[l], v_new[l],
 * k_cache[l], v_cache[l], out[l]: host arrays of n_layers device pointers, each
 * with the layout and rules of bs_dual_cache_block_attention), then K3 on the
 * logits. K3 reads and updates the block cells of the DENSE token and mask
 * boxes directly: tokens / masked are [R][W] with row strides
 * tokens_row_stride / masked_row_stride ELEMENTS (>= W), block cell j of
 * request i at (row_i, off_i + s_i + j). The result equals K1 gather of tokens
 * and mask, K2 per layer, K3 on the compact state, then K1^-1 scatter; only
 * the gather/scatter launches are saved. pos_out ([n][L] int32, may be NULL)
 * receives s_i + j for j < B_i and -1 beyond. conf_out as for K3 ([n][L]).
 * Other arguments as for K2 and K3 (n_layers == 0 runs K3 alone). ws: at
 * least bs_decode_workspace_bytes(n, L, V, logits_dt) bytes (K3's part); with
 * bs_step_workspace_bytes(...) bytes the attention also runs its split-KV
 * plan, its partial slots placed after K3's part rounded up to 256 bytes
 * (see bs_dual_cache_block_attention). All checks run before anything is
 * enqueued.
 */
size_t bs_step_workspace_bytes(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D, bs_dtype dt, int V,
                               bs_dtype logits_dt);
int bs_mixed_state_step(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W, int n_layers, int Hq,
                        int Hkv, int D, bs_dtype dt, float scale, int write_back, const void* const* q,
                        const void* const* k_new, const void* const* v_new, void* const* k_cache,
                        void* const* v_cache, void* const* out, int V, bs_dtype logits_dt, const void* logits,
                        int64_t logits_row_stride, int32_t* tokens, int64_t tokens_row_stride, uint8_t* masked,
                        int64_t masked_row_stride, float tau, int32_t q_min, int32_t eos_id, int32_t* n_unmasked,
                        uint8_t* done, uint8_t* eos_seen, float* conf_out, int32_t* pos_out, void* ws,
                        size_t ws_bytes, void* stream);

/*
 * bs_mixed_state_step for callers that cannot allocate device memory: code
 * under HIP graph capture, serving loops that must not call hipMalloc, and
 * harnesses that forbid allocation. Same arguments, rules and results as
 * bs_mixed_state_step, without the workspace (so every attention row runs
 * whole, no split-KV): the descriptors, the attention
 * work list and the decode partials go to the library's static device array
 * (8 MiB per GPU, held until the process ends), whose address the context
 * resolved when it was created; the call itself allocates nothing and calls
 * no allocating routine. Its host copy of the descriptors goes through one of
 * four pinned stages that bs_create allocated; a call waits for the device
 * only when all four are still being copied from.
 * Limits (BS_ERR_UNSUPPORTED beyond them, before anything is enqueued):
 * n * 20 bytes (rounded up to 16) plus n * Hkv * ceil(L / 32) * 48 bytes of
 * work items (the ceil term only when (Hq / Hkv) * ceil(L / 32) > 8, else 1;
 * no work items for BS_F32 or n_layers == 0) within 512 KiB; bs_decode_workspace_bytes(n, L,
 * V, logits_dt) within 7.5 MiB.
 * Every call on a GPU shares that GPU's array and leaves the last call's
 * contents in it (nothing in it needs to start at zero): calls on one stream
 * are ordered, but calls that may overlap on one GPU (other streams, other
 * contexts or threads) race and must not be issued.
 */
int bs_mixed_state_step_noalloc(bs_ctx* ctx, const bs_req_desc* reqs, int n, int L, int R, int W, int n_layers,
                                int Hq, int Hkv, int D, bs_dtype dt, float scale, int write_back,
                                const void* const* q, const void* const* k_new, const void* const* v_new,
                                void* const* k_cache, void* const* v_cache, void* const* out, int V,
                                bs_dtype logits_dt, const void* logits, int64_t logits_row_stride, int32_t* tokens,
                                int64_t tokens_row_stride, uint8_t* masked, int64_t masked_row_stride, float tau,
                                int32_t q_min, int32_t eos_id, int32_t* n_unmasked, uint8_t* done,
                                uint8_t* eos_seen, float* conf_out, int32_t* pos_out, void* stream);

/*
 * Phase timing of bs_mixed_state_step, bs_lm_head_decode and
 * bs_dual_cache_refresh (a trace facility; no method content).
 * bs_profile_begin arms a ring of max_steps calls: each following call of
 * these entry points records BS_PROFILE_PHASES + 1 HIP events on its stream,
 * until max_steps calls are recorded. For bs_mixed_state_step the phases are
 * attention over all layers, decode row reductions, selection; for
 * bs_lm_head_decode they are the masked-row list, the output-head GEMM with
 * its on-the-fly reduction, and the merge plus selection; for
 * bs_dual_cache_refresh the rotated-key and value scatter, the attention,
 * and an empty third phase. bs_profile_end waits for the recorded events
 * and writes phase_ms[k][ph] (k < *n_steps, ph < BS_PROFILE_PHASES) for up to
 * max_steps calls, then disarms. Events are created once and reused; they
 * are timing-only events (hipEventDisableSystemFence), so a mark adds no
 * cache write-back or invalidation between the phases.
 */
#define BS_PROFILE_PHASES 3
int bs_profile_begin(bs_ctx* ctx, int max_steps);
int bs_profile_end(bs_ctx* ctx, float* phase_ms, int max_steps, int* n_steps);

/* ------------------------------------------------------------------------
 * Host scheduler: block-grained scheduling (Algorithm 1) with compute-aware
 * admission (Section "Compute-aware admission control", Eq. 1). Host memory
 * only; it plans, the step entry points above execute. One block-cycle:
 *   bs_sched_refill  -> descriptors of the active set (row order), the
 *                       admitted requests and the K4 segments that copy their
 *                       staged (prefilled) rows into the box;
 *   the caller runs K4 and then denoising steps until every active block is
 *   fully unmasked;
 *   bs_sched_complete -> every active request advances one block; requests at
 *                       K_i blocks or reporting EOS leave the active set.
 * Queue order, sand filling and the Fixed variant follow the paper; where it
 * is silent: the queue is ascending in p by default (ties: arrival order); a
 * refill alternates two moves until neither admits anything: admit every
 * sand-filling candidate (p + L no wider than the current box) whose
 * admission keeps Eq. 1 within the budget, scanning the whole queue, then
 * admit the head of the queue if it fits (it may widen the box); the Fixed
 * policy admits from the head while fewer than fixed_batch are active. Eq. 1
 * gates admissions only: the rows of admitted requests grow by L per block
 * afterwards, as in Algorithm 1. An admitted request takes
 * the lowest free row, right-aligned at off = width - (p + g).
 * Errors: status codes as above; the detail is in bs_sched_last_error()
 * (thread-local). Not thread-safe per scheduler.
 * ---------------------------------------------------------------------- */
typedef struct bs_sched bs_sched;

enum { BS_SCHED_BUDGET = 0, BS_SCHED_FIXED = 1 };
enum { BS_ORDER_ASCENDING = 0, BS_ORDER_DESCENDING = 1, BS_ORDER_ARRIVAL = 2 };

typedef struct {
  int32_t L;            /* block length */
  int32_t policy;       /* BS_SCHED_BUDGET (Eq. 1 token budget) or BS_SCHED_FIXED (batch cap) */
  int64_t budget;       /* Eq. 1 budget in tokens (budget policy) */
  int32_t fixed_batch;  /* active-set cap (fixed policy) */
  int32_t rows;         /* rows of the physical box (R) */
  int32_t width;        /* columns of the physical box (W) */
  int32_t order;        /* BS_ORDER_*: pending-queue order */
} bs_sched_config;

typedef struct {
  int32_t id;  /* caller's request id (reported back) */
  int32_t p;   /* prompt length */
  int32_t g;   /* generation length */
} bs_sched_request;

/* Filled by bs_sched_refill; the arrays belong to the scheduler and stay valid
 * until its next refill or destroy. */
typedef struct {
  int32_t n_active;             /* active requests after the refill */
  const bs_req_desc* descs;     /* [n_active] descriptors in row order (k = block index) */
  const int32_t* ids;           /* [n_active] request ids, same order */
  int32_t n_admitted;           /* requests admitted by this refill */
  const int32_t* admitted_ids;  /* [n_admitted] in admission order */
  const bs_copy_seg* segs;      /* [n_admitted] staging row a (the a-th admitted request's
                                   prefilled row, left-aligned) -> its row in the box */
  int64_t cost;                 /* Eq. 1 of the active set */
  int32_t box_width;            /* max over the active set of p + (b + 1) L */
} bs_sched_plan;

int bs_sched_create(bs_sched** out, const bs_sched_config* cfg);
int bs_sched_destroy(bs_sched* s);
/* Adds requests to the pending queue. Rejects (BS_ERR_DESCRIPTOR, nothing
 * added) p < 0, g < 1, p + g > width, and under the budget policy p + L >
 * budget (a request that could never be admitted). */
int bs_sched_submit(bs_sched* s, const bs_sched_request* reqs, int n);
int bs_sched_refill(bs_sched* s, bs_sched_plan* plan);
/* End of a block-cycle. eos[i] (may be NULL) flags CheckEOS for the i-th
 * request of the last plan's row order; n must equal the active count.
 * evicted_ids ([n] capacity) receives the ids that left, *n_evicted their
 * number. */
int bs_sched_complete(bs_sched* s, const uint8_t* eos, int n, int32_t* evicted_ids, int32_t* n_evicted);
/* Counters: pending, active, finished, completed block-cycles and the sum of
 * active counts over them (Eq. 2: R = sum_active / (cycles * B)). Any output
 * may be NULL. */
int bs_sched_counts(const bs_sched* s, int32_t* n_pending, int32_t* n_active, int64_t* n_finished,
                    int64_t* cycles, int64_t* sum_active);
const char* bs_sched_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BLOCKSERVE_H */
