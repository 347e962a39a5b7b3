/*
 * eldr_signature.h -- the block-granular expert-signature cache of ELDR
 * (arXiv 2607.00466, Design, Prefix Cache Coherence), for MI355X (gfx950).
 *
 * ELDR routes a request to a decode worker by its expert signature, built
 * from how many of the prompt's tokens the gate sent to each expert at each
 * MoE layer during prefill.  With prefix caching a request's cached blocks are
 * never prefilled again, so the counts are kept per KV-cache block: one row
 * per block, indexed by the block id, one int8 cell per (MoE layer, expert).
 * Prefill adds each token's top-k picks to the row of the block that stores
 * its K/V; a reused block starts from a zero row; a request's counts are the
 * sum of the rows of its blocks, which equals a cold prefill of the same
 * prompt under partial and full prefix hits.
 *
 * Same conventions as eldr_moe.h: plain device pointers, sizes and a
 * hipStream_t passed as void*; the caller owns every buffer; calls are
 * asynchronous on `stream`, allocate nothing, keep no state and never
 * synchronise; they return MOE_OK or a negative MOE_ERR_* code (eldr_moe.h)
 * before any launch.  The cache `sig` is int8 [num_blocks, L, E], row-major,
 * 4-byte aligned, with (L * E) % 4 == 0.
 */
#ifndef ELDR_SIGNATURE_H_
#define ELDR_SIGNATURE_H_

#include <stddef.h>
#include <stdint.h>

#include "eldr_moe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Limits of the signature calls. */
#define MOE_SIG_MAX_LAYERS 1024
#define MOE_SIG_MAX_TOKENS (1 << 20)

/*
 * moe_sig_capture -- add one prefill forward's expert picks to the cache
 * (Design, Prefix Cache Coherence: as prefill writes a token's K/V into a
 * block, the experts the gate picked for that token at each MoE layer are
 * written to the block's row; each forward does this in one GPU pass).
 *
 *   for l < n_layers, t < T, j < K, with b = token_block[t] >= 0:
 *     sig[b, layer0 + l, ids[l, t, j]] += 1
 *
 * ids [n_layers, T, K] int32: the top-k expert ids of the forward's T new
 * tokens at MoE layers layer0 .. layer0 + n_layers - 1 (moe_gate_topk's
 * topk_ids of each layer, stacked).  token_block [T] int32: the KV block each
 * token is written to; a negative entry means the token is not recorded.
 * sig: the cache (in/out).  rejected: NULL, or one int32 on the device that
 * is incremented by the number of picks skipped because the id is outside
 * [0, E) or the block id is >= num_blocks.
 * Cells are int8: a block must receive at most 127 tokens over its lifetime
 * (a KV block size of at most 127).  The counts use exact integer atomics,
 * so the result does not depend on the order of the picks.
 */
int moe_sig_capture(const int32_t* ids, const int32_t* token_block, int32_t n_layers, int32_t T,
                    int32_t K, int32_t layer0, int32_t L, int32_t E, int32_t num_blocks,
                    int8_t* sig, int32_t* rejected, void* stream);

/*
 * moe_sig_reset -- zero the rows of the n blocks listed in `blocks` [n]
 * int32 (blocks handed to a new request start empty, following the KV
 * cache's block lifecycle).  Entries outside [0, num_blocks) are ignored.
 * Uses stores, no memset, so it can be captured in a graph.
 */
int moe_sig_reset(const int32_t* blocks, int32_t n, int32_t L, int32_t E, int32_t num_blocks,
                  int8_t* sig, void* stream);

/*
 * moe_sig_request_counts -- each request's counts: the sum of the rows of
 * the blocks its KV cache spans (Design, Prefix Cache Coherence: s_r is the
 * sum over the request's blocks of sig[b]).
 *
 *   out[r, l, e] = sum over i < n_blocks[r] of sig[block_table[r, i], l, e]
 *
 * block_table [R, max_blocks] int32 and n_blocks [R] int32 (0 <= n_blocks[r]
 * <= max_blocks; entries outside [0, num_blocks) contribute nothing).
 * out [R, L, E] int32 (written in full), ready for one device-to-host copy.
 * int32 keeps the sums exact at any prompt length.
 */
int moe_sig_request_counts(const int8_t* sig, const int32_t* block_table, const int32_t* n_blocks,
                           int32_t R, int32_t max_blocks, int32_t L, int32_t E,
                           int32_t num_blocks, int32_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif  /* ELDR_SIGNATURE_H_ */
