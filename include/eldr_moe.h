/*
 * eldr_moe.h -- C ABI of the MI355X (gfx950) batched-decode MoE layer.
 *
 * The layer is the computation that ELDR's expert-locality routing speeds up
 * (Introduction; Motivation, "Active Expert Count Drives MoE Decode Latency"):
 * in a decode step every token is scored by the MoE gate, dispatched to its
 * top-k experts, and the step must fetch from HBM the weights of every
 * distinct expert the batch activates -- the union -- and nothing else.
 * ELDR changes only which worker serves a request, so the layer itself is
 * standard top-k gating (Introduction; Related Work) and this library computes
 * exactly that, in four calls run back to back on one stream:
 *
 *   moe_gate_topk   gate scores, top-k selection and renormalised weights
 *   moe_bucket      per-expert buckets and the distinct-expert union
 *   moe_expert_ffn  SwiGLU FFN of every expert in the union, on its tokens
 *   moe_combine     weighted sum of each token's k expert outputs
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every pointer argument except `stream` is a DEVICE pointer owned by the
 *   caller; the library allocates nothing and keeps no state between calls.
 *   `stream` is a hipStream_t passed as void* (NULL = the null stream).
 * - Calls are asynchronous on `stream` and never synchronise.  Device faults
 *   surface at the caller's next synchronisation.
 * - Return value: MOE_OK (0) after a successful launch, or a negative status
 *   (below) when arguments are rejected before anything is launched, or
 *   MOE_ERR_HIP when the runtime reports a launch error.  Nothing aborts,
 *   throws or exits across this boundary.
 * - Layouts are row-major.  Float data is IEEE binary32 ("fp32").  bf16 data
 *   is passed as raw 16-bit patterns (uint16_t), the upper half of a binary32.
 * - Weights are defined row-major [out, in] (each output neuron's weights
 *   contiguous along the reduction axis):
 *     w_gate [E, H] fp32; w1, w3 [E, I, H] bf16; w2 [E, H, I] bf16.
 *   The math is y = W2 (silu(W1 x) * (W3 x)) with silu(z) = z / (1 + e^-z).
 *   The expert FFN takes the expert weights *packed* by moe_pack_up_weights
 *   (w1 with w3) and moe_pack_down_weights (w2), a permutation done once,
 *   when the model is loaded (see below).
 * - Pointers to fp32 or bf16 arrays must be 16-byte aligned (the kernels use
 *   128-bit loads and stores); int32 arrays 4-byte aligned.
 * - T = 0 (an empty batch) is accepted everywhere: nothing is computed except
 *   that moe_bucket still writes empty buckets and a zero union.
 */
#ifndef ELDR_MOE_H
#define ELDR_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Shape of one layer invocation: T tokens, hidden size H, E experts, top-K,
 * expert intermediate size I. */
typedef struct moe_dims {
  int32_t T, H, E, K, I;
} moe_dims;

/* Status codes. */
#define MOE_OK 0
#define MOE_ERR_INVALID (-1)     /* null pointer, negative size, K > E, ...   */
#define MOE_ERR_UNSUPPORTED (-2) /* shape outside the limits below, bad alignment */
#define MOE_ERR_WORKSPACE (-3)   /* workspace smaller than *_workspace_bytes  */
#define MOE_ERR_HIP (-4)         /* the HIP runtime rejected the launch       */

/* Limits.  H and I must be multiples of 32 (one MFMA reduction step). */
#define MOE_MAX_E 256
#define MOE_MAX_K 16
#define MOE_MAX_T 4096
#define MOE_MAX_H 16384
#define MOE_MAX_I 16384

/* Human-readable name of a status code (static storage, never NULL). */
const char* moe_status_string(int status);

/* Version of this ABI (bumped on any incompatible change). */
int moe_abi_version(void);

/*
 * moe_gate_topk -- the MoE gate (Introduction: the gate picks each token's
 * experts from its hidden representation; Design, Signature Design: scores
 * are computed for all E experts, only the discrete top-k fetch one).
 *
 *   logits[t, e] = sum_h x[t, h] * w_gate[e, h]        (fp32 accumulation)
 *   topk_ids[t, :] = the K experts with the largest logits, in descending
 *                    logit order; equal logits go to the lower expert id
 *   topk_w[t, j]   = softmax(logits[t, :])[id] / sum over the K picks
 *                  = exp(l_j - l_max) / sum_j' exp(l_j' - l_max)
 *
 * x [T, H] fp32, w_gate [E, H] fp32 (inputs).  logits [T, E] fp32,
 * topk_ids [T, K] int32, topk_w [T, K] fp32 (outputs, all written).
 * Every expert's score is reduced in the same order, so experts with
 * identical gate rows tie exactly and the lower id wins; that order depends
 * on H alone, so a token's logits, ids and weights are the same bits in any
 * batch.  Inputs must be finite.
 */
int moe_gate_topk(const float* x, const float* w_gate, moe_dims d, float* logits,
                  int32_t* topk_ids, float* topk_w, void* stream);

/*
 * moe_bucket -- group the batch's (token, expert) pairs by expert and form
 * the distinct-expert union whose weights the step must load (Motivation,
 * "Active Expert Count Drives MoE Decode Latency").
 *
 * topk_ids [T, K] int32 (input): ids in [0, E), distinct within a token.
 * Outputs (all written):
 *   counts     [E]     tokens per expert
 *   offsets    [E+1]   exclusive prefix sum of counts; offsets[E] = T*K
 *   perm_token [T*K]   token of each slot: experts ascending, and within an
 *                      expert tokens ascending
 *   pair_pos   [T*K]   pair_pos[t*K + j] = slot of (t, topk_ids[t, j])
 *   union_ids  [2E]    the union twice: [0, E) the experts with counts > 0
 *                      ascending, then -1 padding; [E, 2E) the same experts
 *                      in dispatch order -- more 16-token tiles
 *                      (ceil(count / 16)) first, equal ones by ascending id --
 *                      then -1 padding (moe_expert_ffn runs the largest
 *                      buckets first and deals experts to XCDs in this order)
 *   union_size [1]     number of distinct experts U (stays on the device)
 * If an id is out of range or repeated within a token, union_size is set to
 * -1 and the other outputs are unspecified; moe_expert_ffn then does nothing.
 * Requires E * ceil(T / 32) <= 16384 (per-expert token bitmaps in LDS),
 * else MOE_ERR_UNSUPPORTED; above 8192 it raises the kernel's dynamic LDS
 * limit on the current device first (MOE_ERR_HIP if the runtime refuses).
 */
int moe_bucket(const int32_t* topk_ids, moe_dims d, int32_t* counts, int32_t* offsets,
               int32_t* perm_token, int32_t* pair_pos, int32_t* union_ids,
               int32_t* union_size, void* stream);

/*
 * moe_pack_up_weights / moe_pack_down_weights -- lay the bf16 expert weights
 * out as the expert FFN streams them.  Call once per layer, off the decode
 * path (when the model is loaded); asynchronous on `stream`.
 *
 * The FFN reads 16-row x 32-column tiles as MFMA A fragments: lane l
 * (0..63) takes row l % 16 and the 8 values starting at column 8 (l / 16).
 * One fragment is 1 KB, its 64 lane pieces in lane order.  A workgroup item
 * is a band of rows -- up: 64 rows of W1 and the same 64 rows of W3; down:
 * 128 rows of W2 -- handled by 4 waves, each reading two fragments per
 * k-step of 32 values: up wave w: rows 16 w .. 16 w + 15 of the band, of W1
 * then W3; down wave w: rows 32 w .. 32 w + 15, then 32 w + 16 .. 32 w + 31.
 * The packed order is, for each expert, band, k-step, wave (w ascending)
 * and its two fragments, the fragment's 64 lane pieces, so that one item is
 * one contiguous stretch of memory.  A last band with fewer rows (R not a
 * multiple of the band) holds only its waves' fragments.
 *
 *   moe_pack_up_weights:   w1, w3 [E, I, H] -> w13, 2 * E * I * H bf16
 *   moe_pack_down_weights: w2 [E, H, I]     -> w2p, E * H * I bf16
 *
 * Values are unchanged (a permutation).  Inputs and output are distinct
 * 16-byte-aligned device buffers; I % 32 == 0 and H % 32 == 0 (else
 * MOE_ERR_UNSUPPORTED).
 */
int moe_pack_up_weights(const uint16_t* w1, const uint16_t* w3, int32_t E, int32_t I, int32_t H,
                        uint16_t* w13, void* stream);
int moe_pack_down_weights(const uint16_t* w2, int32_t E, int32_t H, int32_t I, uint16_t* w2p,
                          void* stream);

/* Bytes of device workspace moe_expert_ffn needs for dims d: the SwiGLU
 * activations of every slot, stored as pairs of bf16 values (4 bytes a
 * value): 4 * T*K*I.  0 when T == 0. */
size_t moe_ffn_workspace_bytes(moe_dims d);

/*
 * moe_expert_ffn -- the expert FFNs of the union (Motivation: each step
 * fetches the weights of every expert the batch activates; Introduction:
 * weight reuse happens only among tokens sharing an expert).
 *
 * For every u < union_size, with e = union_ids[u] and its slots
 * s in [offsets[e], offsets[e+1]) holding token t = perm_token[s]:
 *   y_perm[s, :] = W2_e (silu(W1_e x[t]) * (W3_e x[t]))
 * Each active expert's weights are streamed from HBM once per call when its
 * bucket fits one token group: the whole batch when T <= 64, else 128
 * tokens; a bigger bucket is split into groups of 128 tokens whose
 * workgroups run side by side on one XCD and share that XCD's L2 for the
 * repeated weight reads.  Experts outside the union are never touched.
 * Work follows the union's dispatch order (largest buckets first): with
 * T <= 64 experts are dealt round-robin over the 8 XCDs, with T > 64 their
 * (expert, row band) units are, so skewed buckets still load the XCDs evenly.
 * The grid is sized from E and T alone and reads union_size on the device,
 * so no host synchronisation is needed between moe_bucket and this call.
 *
 * x [T, H] fp32; w13 (W1 and W3, [E, I, H] each) packed by
 * moe_pack_up_weights and w2 ([E, H, I]) packed by moe_pack_down_weights;
 * offsets [E+1],
 * perm_token [T*K], union_ids [2E], union_size [1] int32 (moe_bucket output;
 * the FFN reads the dispatch-order half of union_ids).
 * y_perm [T*K, H] fp32 output (rows of slots whose expert is not in the
 * union are not written).  ws: device workspace of at least
 * moe_ffn_workspace_bytes(d) bytes, 16-byte aligned, contents irrelevant.
 * Arithmetic: bf16 weights times activations carried as a pair of bf16
 * values (high part and rounded remainder, about 16 significant bits) on
 * MFMA with fp32 accumulation.  Every pass shape accumulates a slot's
 * products in the same k order, so y_perm[s, :] depends on its token's x
 * and its expert's weights alone: the same bits whatever else is in the
 * batch (and likewise for the MXFP4, routed and fused forms).
 */
int moe_expert_ffn(const float* x, const uint16_t* w13, const uint16_t* w2,
                   const int32_t* offsets, const int32_t* perm_token, const int32_t* union_ids,
                   const int32_t* union_size, moe_dims d, float* y_perm, void* ws,
                   size_t ws_bytes, void* stream);

/*
 * The two halves of moe_expert_ffn, for callers that time or schedule them
 * separately (moe_expert_ffn is exactly up followed by down on one stream).
 *
 * moe_expert_ffn_up: for every slot s of an expert e in the union, the
 *   activation h_s = silu(W1_e x[t]) * (W3_e x[t]), t = perm_token[s], is
 *   left in the workspace (as a pair of bf16 values per element).
 * moe_expert_ffn_down: y_perm[s, :] = W2_e h_s, reading h from the workspace.
 * Arguments, layouts, the workspace size and error behaviour are those of
 * moe_expert_ffn; ws_bytes is the size of the workspace `ws`, which must be
 * the one the preceding moe_expert_ffn_up call filled.
 */
int moe_expert_ffn_up(const float* x, const uint16_t* w13, const int32_t* offsets,
                      const int32_t* perm_token, const int32_t* union_ids,
                      const int32_t* union_size, moe_dims d, void* ws, size_t ws_bytes,
                      void* stream);
int moe_expert_ffn_down(const void* ws, const uint16_t* w2, const int32_t* offsets,
                        const int32_t* perm_token, const int32_t* union_ids,
                        const int32_t* union_size, moe_dims d, size_t ws_bytes, float* y_perm,
                        void* stream);

/*
 * moe_expert_ffn_noalloc -- moe_expert_ffn without a caller workspace, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The workspace (h of
 * every slot, moe_ffn_workspace_bytes(d) bytes) lives in a fixed device array
 * of moe_expert_ffn_noalloc_max_bytes() = 32 MiB inside the library, one per
 * GPU, held until the process ends; its address is taken on the first call on
 * each device.  The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine).  Arguments, layouts, results and errors as
 * moe_expert_ffn; a problem whose workspace exceeds 32 MiB (T*K*I*4 bytes)
 * returns MOE_ERR_WORKSPACE before any launch.  Every call on one GPU shares
 * that GPU's array, which keeps the last call's contents (nothing in it needs
 * to start at zero): calls that overlap on one GPU -- on different streams,
 * or from different host threads without ordering -- race and must not be
 * made.
 */
int moe_expert_ffn_noalloc(const float* x, const uint16_t* w13, const uint16_t* w2,
                           const int32_t* offsets, const int32_t* perm_token,
                           const int32_t* union_ids, const int32_t* union_size, moe_dims d,
                           float* y_perm, void* stream);
size_t moe_expert_ffn_noalloc_max_bytes(void);

/*
 * moe_expert_ffn_up_routed -- moe_bucket followed by moe_expert_ffn_up, in
 * one launch for batches of at most 64 tokens (two launches above that).
 * The step after the gate (Motivation, "Active Expert Count Drives MoE Decode
 * Latency": the union of the batch's picks is what the step loads) and the
 * first half of the expert FFN, fused so that no separate bucketing launch
 * sits between the routing and the weight stream: every workgroup of the up
 * projection builds the buckets of the routing in its own LDS, and one of
 * them also writes moe_bucket's outputs for moe_expert_ffn_down and
 * moe_combine.
 *
 * topk_ids [T, K] int32 (input, as for moe_bucket); counts, offsets,
 * perm_token, pair_pos, union_ids, union_size (outputs, identical to
 * moe_bucket's, bit for bit, invalid routing included); x, w13, ws,
 * ws_bytes as for moe_expert_ffn_up, whose workspace result it leaves.
 * Errors as moe_bucket and moe_expert_ffn_up; nothing is launched on an
 * error.
 */
int moe_expert_ffn_up_routed(const float* x, const uint16_t* w13, const int32_t* topk_ids,
                             moe_dims d, int32_t* counts, int32_t* offsets, int32_t* perm_token,
                             int32_t* pair_pos, int32_t* union_ids, int32_t* union_size,
                             void* ws, size_t ws_bytes, void* stream);

/*
 * moe_expert_ffn_routed -- moe_bucket followed by moe_expert_ffn, in one
 * launch for batches of at most 64 tokens (the separate calls above that).
 * The whole expert step of a decode batch after the gate (Motivation,
 * "Active Expert Count Drives MoE Decode Latency": the union of the batch's
 * picks is what the step loads): every workgroup builds the buckets of the
 * routing in its own LDS, as in moe_expert_ffn_up_routed; an XCD's workgroups
 * take the up bands of its experts first, then their down bands, and a down
 * band waits on the device until every up band of its expert has stored h,
 * so the down projection's weights start streaming while the up projection
 * ends, with no launch between them.
 *
 * topk_ids [T, K] int32 (input); counts, offsets, perm_token, pair_pos,
 * union_ids, union_size (outputs, moe_bucket's, bit for bit); x, w13, w2,
 * y_perm, ws, ws_bytes as for moe_expert_ffn, whose y_perm (and workspace)
 * results it leaves, bit for bit; ws must be 128-byte aligned here (else
 * MOE_ERR_UNSUPPORTED).
 * sync: int32 [64 E + 1] (moe_ffn_sync_bytes), caller-owned device memory
 * that must be zero before the first call; every call leaves it zero.  Words
 * 0 .. 64E-1 hold two counters per union position, one 256-byte line each (so
 * that the waits' polls spread over memory channels); word 64E becomes 1 if a
 * down band gave up waiting for its expert (a bounded wait of about 2^18
 * polls that a correct run never reaches: the GPU starts an XCD's
 * workgroups in index order and every up band precedes every down band of
 * its XCD), in which case that call's y_perm is not valid and the counters
 * must be zeroed again before the next call.  Calls that share one `sync`
 * buffer must not overlap (one stream, or ordered by events); calls with
 * different buffers may.  Errors as moe_bucket and moe_expert_ffn, plus
 * MOE_ERR_INVALID for a null sync and MOE_ERR_UNSUPPORTED for a misaligned
 * one; nothing is launched on an error.
 */
int moe_expert_ffn_routed(const float* x, const uint16_t* w13, const uint16_t* w2,
                          const int32_t* topk_ids, moe_dims d, int32_t* counts, int32_t* offsets,
                          int32_t* perm_token, int32_t* pair_pos, int32_t* union_ids,
                          int32_t* union_size, float* y_perm, void* ws, size_t ws_bytes,
                          int32_t* sync, void* stream);
/* Bytes of moe_expert_ffn_routed's sync buffer: 4 (64 E + 1); 0 for invalid dims. */
size_t moe_ffn_sync_bytes(moe_dims d);

/*
 * MXFP4 expert weights (Evaluation, "Models": GPT-OSS-120B is served in
 * mxfp4).  The format is the OCP Microscaling (MX) v1.0 MXFP4: blocks of 32
 * values along the reduction axis share one E8M0 scale X = 2^(code - 127);
 * each value is an FP4 E2M1 code (sign, 2-bit exponent with bias 1, 1-bit
 * mantissa: magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6) and stands for X times
 * its magnitude.  Unpacked tensors, as checkpoints store them:
 *   codes  [E, R, K/2] uint8, value k of a row in byte k/2, the even k in
 *          the low nibble;
 *   scales [E, R, K/32] uint8, the scale of values 32 j .. 32 j + 31 at j.
 * Scale codes must lie in 1 .. 252 (every dequantized value is then a finite
 * bf16 number); 0, 253 .. 255 are not supported and are not checked.
 *
 * moe_pack_mxfp4_up / moe_pack_mxfp4_down -- permute the unpacked W1 and W3
 * ([E, I, H]) or W2 ([E, H, I]) into the layout the MXFP4 FFN streams, once,
 * off the decode path.  A wave band is 16 rows of W1 and the same 16 rows of
 * W3 (up), or 32 rows of W2 (down); a workgroup band is 4 consecutive wave
 * bands (the last one of an expert may hold fewer).  A slot s is two k-steps
 * (64 values: H/64 slots up, I/64 down).  For each expert, workgroup band,
 * slot, wave band within it and lane l (0 .. 63), 16 bytes: the 4 code bytes
 * of row l % 16 and values 64 s + 8 (l / 16) .. + 7, then the same for
 * 64 s + 32 + 8 (l / 16), of tile 0 (up: W1; down: the wave band's first 16
 * rows), then both again for tile 1 (up: W3; down: its last 16 rows).
 * Scales: in the same (expert, workgroup band, slot, wave band) order, 16
 * dwords (row 0 .. 15), each the 4 scale bytes in that same order.  A
 * workgroup item thus reads one contiguous stretch of codes and one of
 * scales.  codes receives E*I*H bytes (up) or
 * E*H*I/2 (down), scales E*I*H/16 (up) or E*H*I/32 (down): the unpacked
 * sizes.  Inputs and outputs are distinct device buffers; code inputs and
 * scale outputs 4-byte aligned, code outputs 16-byte aligned.  Requires
 * H % 64 == 0 and I % 64 == 0.  Asynchronous on `stream`.
 */
int moe_pack_mxfp4_up(const uint8_t* w1_codes, const uint8_t* w1_scales, const uint8_t* w3_codes,
                      const uint8_t* w3_scales, int32_t E, int32_t I, int32_t H, uint8_t* codes,
                      uint8_t* scales, void* stream);
int moe_pack_mxfp4_down(const uint8_t* w2_codes, const uint8_t* w2_scales, int32_t E, int32_t H,
                        int32_t I, uint8_t* codes, uint8_t* scales, void* stream);

/*
 * moe_expert_ffn_mxfp4 -- moe_expert_ffn with MXFP4 expert weights, packed by
 * moe_pack_mxfp4_up (up_codes, up_scales) and moe_pack_mxfp4_down
 * (down_codes, down_scales):
 *   y_perm[s, :] = W2_e (silu(W1_e x[t]) * (W3_e x[t]))
 * with every W the dequantized matrix.  The codes are expanded to bf16 in
 * registers (exact: an E2M1 value times a power of two in range is a bf16
 * number) and multiplied exactly as in moe_expert_ffn, so the result equals
 * moe_expert_ffn's on the dequantized weights.  Each active expert's codes
 * and scales are streamed once per call when its bucket fits one token group
 * (the whole batch when T <= 64, else 32 tokens); a bigger bucket is split
 * into groups of 32 tokens sharing the XCD's L2.
 * Other arguments, the workspace (moe_ffn_workspace_bytes) and the error
 * behaviour are those of moe_expert_ffn; in addition H % 64 == 0 and
 * I % 64 == 0 (else MOE_ERR_UNSUPPORTED), and the scale pointers must be
 * 4-byte aligned.  _up and _down are its two halves, as for moe_expert_ffn.
 */
int moe_expert_ffn_mxfp4(const float* x, const uint8_t* up_codes, const uint8_t* up_scales,
                         const uint8_t* down_codes, const uint8_t* down_scales,
                         const int32_t* offsets, const int32_t* perm_token,
                         const int32_t* union_ids, const int32_t* union_size, moe_dims d,
                         float* y_perm, void* ws, size_t ws_bytes, void* stream);
int moe_expert_ffn_mxfp4_up(const float* x, const uint8_t* up_codes, const uint8_t* up_scales,
                            const int32_t* offsets, const int32_t* perm_token,
                            const int32_t* union_ids, const int32_t* union_size, moe_dims d,
                            void* ws, size_t ws_bytes, void* stream);
int moe_expert_ffn_mxfp4_down(const void* ws, const uint8_t* down_codes,
                              const uint8_t* down_scales, const int32_t* offsets,
                              const int32_t* perm_token, const int32_t* union_ids,
                              const int32_t* union_size, moe_dims d, size_t ws_bytes,
                              float* y_perm, void* stream);
/* moe_expert_ffn_mxfp4_up_routed -- moe_expert_ffn_up_routed with MXFP4
 * weights (up_codes, up_scales as for moe_expert_ffn_mxfp4_up). */
int moe_expert_ffn_mxfp4_up_routed(const float* x, const uint8_t* up_codes,
                                   const uint8_t* up_scales, const int32_t* topk_ids, moe_dims d,
                                   int32_t* counts, int32_t* offsets, int32_t* perm_token,
                                   int32_t* pair_pos, int32_t* union_ids, int32_t* union_size,
                                   void* ws, size_t ws_bytes, void* stream);
/* moe_expert_ffn_mxfp4_routed -- moe_expert_ffn_routed with MXFP4 weights
 * (up_codes, up_scales, down_codes, down_scales as for moe_expert_ffn_mxfp4;
 * H % 64 == 0 and I % 64 == 0). */
int moe_expert_ffn_mxfp4_routed(const float* x, const uint8_t* up_codes, const uint8_t* up_scales,
                                const uint8_t* down_codes, const uint8_t* down_scales,
                                const int32_t* topk_ids, moe_dims d, int32_t* counts,
                                int32_t* offsets, int32_t* perm_token, int32_t* pair_pos,
                                int32_t* union_ids, int32_t* union_size, float* y_perm, void* ws,
                                size_t ws_bytes, int32_t* sync, void* stream);

/*
 * moe_combine -- weighted unpermute: out[t, :] = sum over j = 0..K-1 (in that
 * order) of topk_w[t, j] * y_perm[pair_pos[t*K + j], :].  This is the last
 * step of the MoE layer: a token's output is its selected experts' outputs
 * mixed by the gate's renormalised weights (Background, Mixture-of-Experts
 * LLMs; standard top-k gating, which ELDR leaves unchanged: Related Work,
 * "lossless").  Deterministic, no atomics.  y_perm [T*K, H], topk_w [T, K] fp32, pair_pos [T*K] int32
 * (inputs); out [T, H] fp32 (output).  A pair_pos entry outside [0, T*K)
 * contributes nothing.
 */
int moe_combine(const float* y_perm, const int32_t* pair_pos, const float* topk_w, moe_dims d,
                float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ELDR_MOE_H */
