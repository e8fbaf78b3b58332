/*
 * pic_cache.h -- block hashing and span-cache lookup of libpic_attn.so (host only).
 *
 * The other half of the engine change next to the position-free cache (MiniPIC,
 * Sec. 3.1.1 "Three User-Facing Primitives", eq. (1)): every full KV block of a
 * token sequence gets a hash chained through the preceding block, except that a
 * block whose FIRST token is the span-separator token starts a new chain from the
 * seed, and a block whose first token is the prompt-depend token hashes the whole
 * prefix up to and including itself:
 *
 *     h_i = H(h_0, x_i)        if x_i starts with SSEP
 *           H(h_0, x_{<=i})    if x_i starts with PDEP
 *           H(h_{i-1}, x_i)    otherwise
 *
 * with h_0 a 32-byte seed and H = SHA-256 (FIPS 180-4) over the 32-byte chaining
 * value followed by the block tokens as int32 little-endian; for the PDEP case the
 * tokens are those of blocks 0..i.  A trailing partial block is never hashed (it
 * cannot be reused).  A block that hits in the cache can be attended to at any
 * offset without recomputation because the pool holds unrotated keys (Sec. 3.2).
 *
 * Conventions: as in pic_attn.h -- every call returns a pic_status, arguments are
 * checked first and pic_last_error() explains a failure; all arrays are HOST memory
 * owned by the caller.  None of these functions touches the GPU.
 */
#ifndef PIC_CACHE_H
#define PIC_CACHE_H

#include <stddef.h>
#include <stdint.h>

#include "pic_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* SHA-256 of `bytes` bytes at `data` into out[32] (exposed for testing). */
pic_status pic_sha256(const void* data, size_t bytes, uint8_t* out);

/* Hashes of the n_tokens / 16 full blocks of `tokens` (HOST [n_tokens]) by eq. (1):
 * out (HOST [n_tokens/16][32]).  seed: HOST [32] (h_0).  ssep_token / pdep_token
 * are the two marker token ids (they may be any int32 values, but must differ). */
pic_status pic_block_hashes(const int32_t* tokens, int32_t n_tokens, int32_t ssep_token, int32_t pdep_token,
                            const uint8_t* seed, uint8_t* out);

/* Span structure of a token sequence for pic_attn_prefill, given which full blocks
 * hit in the cache (hit: HOST [n_tokens/16], nonzero = cached).  A span starts at
 * token 0, at every block whose first token is a marker (flag PIC_SSEP or PIC_PDEP)
 * and at the first missed block after a cached block of the same chain (no marker
 * flag: it continues the chain's window).  Spans holding missed blocks, or the
 * trailing partial block, carry PIC_QUERY: they are computed in the call; the
 * others are read from the cache.  Writes up to `capacity` spans to span_start /
 * span_flags (HOST) and the count to *n_spans (PIC_EINVAL if capacity is short). */
pic_status pic_spans_from_blocks(const int32_t* tokens, int32_t n_tokens, int32_t ssep_token,
                                 int32_t pdep_token, const uint8_t* hit, int32_t* span_start,
                                 int32_t* span_flags, int32_t capacity, int32_t* n_spans);

/* A host map from block hash to physical block id (the span cache).  Owned by the
 * caller through the handle; not thread-safe (one handle per thread, or lock). */
typedef struct pic_block_cache pic_block_cache;

pic_status pic_block_cache_create(pic_block_cache** cache);
pic_status pic_block_cache_destroy(pic_block_cache* cache);
/* block_ids[i] = cached block of hashes[i] (HOST [n][32]) or -1 on a miss; *n_hits
 * (may be NULL) = number of hits. */
pic_status pic_block_cache_lookup(const pic_block_cache* cache, const uint8_t* hashes, int32_t n,
                                  int32_t* block_ids, int32_t* n_hits);
/* Record hashes[i] -> block_ids[i] (entries with block_ids[i] < 0 are skipped; an
 * existing hash keeps its block). */
pic_status pic_block_cache_insert(pic_block_cache* cache, const uint8_t* hashes, const int32_t* block_ids,
                                  int32_t n);
/* Forget hashes[i] (eviction by the caller); unknown hashes are ignored. */
pic_status pic_block_cache_erase(pic_block_cache* cache, const uint8_t* hashes, int32_t n);
pic_status pic_block_cache_size(const pic_block_cache* cache, int32_t* size);

#ifdef __cplusplus
}
#endif

#endif /* PIC_CACHE_H */
