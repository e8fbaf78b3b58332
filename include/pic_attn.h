/*
 * pic_attn.h -- position-free paged attention on MI355X (gfx950).
 *
 * C ABI of libpic_attn.so.  The operation is the attention step of a KV cache
 * that stores keys without positional rotation (MiniPIC, Sec. 3.2.1 "Mechanism"):
 * RoPE is applied inside the kernel to the queries and to every K tile at the
 * token's per-request logical position, and the visible keys of each query follow
 * the span structure that the SSep / PDep primitives and block-aligned padding
 * define (Sec. 3.1.1, eq. (1)).  The score of query t and cached key j is
 *     (R_{p(t)} q_t)^T (R_{p(j)} k~_j) * scale
 * where k~ is the stored (unrotated) key and p(.) the request's logical position.
 *
 * Conventions shared by every entry point
 *  - Every call returns a pic_status.  Arguments are validated on the host before
 *    anything is enqueued; on an error nothing is launched and pic_last_error()
 *    returns a message (thread-local, valid until the next call on that thread).
 *  - Device contents (block ids, positions, slot numbers) are trusted, as the
 *    paper keeps validation outside the engine (Sec. 3.1.2).  Out-of-range block
 *    ids or slots are undefined behaviour.
 *  - "DEVICE" pointers are HIP device memory; "HOST" pointers are host memory read
 *    during the call only.  All buffers are owned by the caller; the library
 *    allocates nothing and keeps no state between calls (the one exception is the
 *    per-GPU device scratch of pic_attn_decode_noalloc, described there).
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t, or NULL for the
 *    null stream).  Kernel execution errors surface at the caller's next sync.
 *  - Tensors are dense and row-major in the shapes given.  Q, O, the K/V pools
 *    and new K/V rows share cfg->dtype.
 *  - Tensors (Q, O, pools, new rows, rope tables, the workspace) start on 16-byte
 *    boundaries and int32 arrays on 4-byte boundaries; other addresses are
 *    rejected with PIC_EINVAL before anything is launched.
 */
#ifndef PIC_ATTN_H
#define PIC_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pic_status;
#define PIC_OK 0
#define PIC_EINVAL 1       /* malformed argument (null pointer, bad shape, bad span list) */
#define PIC_EUNSUPPORTED 2 /* well formed but not implemented (e.g. head_dim 96) */
#define PIC_EHIP 3         /* a HIP runtime call or launch failed */
#define PIC_EWORKSPACE 4   /* workspace smaller than pic_workspace_size() asked for */

/* element types (cfg->dtype) */
#define PIC_BF16 0
#define PIC_F32 1

/* RoPE pairing (cfg->rope_style).  The paper uses the model's rotary embedding
 * (Sec. 3.2.1) without naming a pairing; NeoX (element i with i + D/2, the
 * Llama convention) is the default, GPT-J (2i with 2i+1) the alternative. */
#define PIC_ROPE_NEOX 0
#define PIC_ROPE_GPTJ 1

/* span flags (span_flags[]), Sec. 3.1.1:
 *  PIC_SSEP  the span is detached from what precedes it: it sees only itself;
 *  PIC_PDEP  the span depends on the whole preceding prompt: it sees everything;
 *  neither   the span continues the previous span's hash chain and keeps its window;
 *  PIC_QUERY the span's tokens are computed in this prefill call (they are the
 *            query rows of q and o). */
#define PIC_SSEP 1
#define PIC_PDEP 2
#define PIC_QUERY 4

typedef struct pic_config {
    int32_t num_q_heads;   /* Hq > 0 */
    int32_t num_kv_heads;  /* Hkv > 0, Hq % Hkv == 0; query head h reads KV head h / (Hq/Hkv) */
    int32_t head_dim;      /* D: 64 or 128 */
    int32_t block_size;    /* tokens per KV block: must be 16 */
    int32_t dtype;         /* PIC_BF16 or PIC_F32 */
    int32_t rope_style;    /* PIC_ROPE_NEOX or PIC_ROPE_GPTJ */
    double rope_theta;     /* base of omega_i = theta^(-2i/D), > 0 */
    float softmax_scale;   /* 0 means 1/sqrt(D) (Sec. 3.2.1 score equation) */
    int32_t k_prerotated;  /* 0: the pool holds unrotated K and q is unrotated (the method);
                              1: both are already rotated and no RoPE is applied (the
                                 baseline FlashAttention of Sec. 3.2.2, for comparison) */
    /* RoPE variants of the models the method applies to (Sec. 3.2.1 takes the model's
     * own rotary embedding).  rotary_dim R: only the first R elements of q and k turn
     * (partial rotary), 0 means R = D; even, 2 <= R <= D.  Within them PIC_ROPE_GPTJ
     * pairs 2i with 2i+1 and PIC_ROPE_NEOX pairs i with i + R/2 (NeoX with R < D
     * needs R % 16 == 0, else PIC_EUNSUPPORTED).  inv_freq: HOST [R/2] frequencies
     * omega_i (radians per position), finite, read during each call that takes cfg --
     * scaled-RoPE variants (position interpolation, NTK, Llama-3-style band scaling)
     * change only these; NULL means omega_i = theta^(-2i/R). */
    const double* inv_freq;
    int32_t rotary_dim;
} pic_config;

/* Span structure of a batch (HOST).  Request r has seq_lens[r] >= 1 tokens
 * (cached and new) indexed n = 0..L_r-1 and spans cu_spans[r] .. cu_spans[r+1]-1
 * (at least one).  span_start[] is 0 for a request's first span and strictly
 * increasing.  span_window, if not NULL, holds an explicit window start per span
 * (-1: use the flags), with 0 <= w <= span start; it generalises SSep/PDep. */
typedef struct pic_batch_host {
    int32_t num_reqs;
    const int32_t* seq_lens;    /* HOST [R] */
    const int32_t* cu_spans;    /* HOST [R+1], cu_spans[0] == 0 */
    const int32_t* span_start;  /* HOST [S] */
    const int32_t* span_flags;  /* HOST [S] */
    const int32_t* span_window; /* HOST [S] or NULL */
} pic_batch_host;

/* Per-token metadata (DEVICE).  Token n of request r lives in physical block
 * block_tables[r*max_blocks + n/16] at offset n%16; its logical position (only fed
 * to RoPE, never to the mask) is positions[sum_{r'<r} L_r' + n].  A physical block
 * may appear in many requests and more than once in one request. */
typedef struct pic_batch_dev {
    const int32_t* block_tables; /* DEVICE [R][max_blocks] */
    int32_t max_blocks;          /* >= ceil(L_r / 16) for every r */
    const int32_t* positions;    /* DEVICE [sum L_r], any int32 values */
} pic_batch_dev;

/* Optional cos/sin table (the paper's cos_sin lookup, Sec. 3.2.2): one entry per
 * (position p in [0, len), pair i in [0, D/2)), from cos/sin(p*omega_i) computed in
 * float64 (omega_i = 0 for pairs past rotary_dim).  A table belongs to the
 * frequencies of the cfg that built it.  PIC_F32 tables hold (cos, sin) as two
 * float32 (8 bytes per entry); PIC_BF16 tables hold (cos, sin) as a bf16 pair (4
 * bytes), with which the kernel rotates a pair (x, y) by two 2-element dot products.
 * Built by pic_rope_table_build for cfg->dtype; pic_rope_table_bytes gives the size.
 * Positions outside [0, len), and every position when data is NULL, are rotated
 * with cos/sin computed in the kernel from an exact fixed-point phase. */
typedef struct pic_rope_table {
    const void* data; /* DEVICE [len][D/2] entries (8 bytes for PIC_F32, 4 for PIC_BF16), or NULL */
    int32_t len;
} pic_rope_table;

/* Library version (major*10000 + minor*100 + patch). */
int32_t pic_version(void);

/* Message of the last error on this thread ("" if none). */
const char* pic_last_error(void);

/* Bytes of the cos/sin table for positions [0, num_positions). */
pic_status pic_rope_table_bytes(const pic_config* cfg, int32_t num_positions, size_t* bytes);

/* Fill `table` (DEVICE, pic_rope_table_bytes bytes) with the entries of positions
 * [0, num_positions) in the format of cfg->dtype (see pic_rope_table). */
pic_status pic_rope_table_build(const pic_config* cfg, int32_t num_positions, void* table, void* stream);

/* Rotate x (DEVICE [n][num_heads][D], cfg->dtype) in place by R_p with
 * p = positions[i] (DEVICE [n]) for row i.  This is the conventional
 * rotary-embedding step; it builds the pre-rotated inputs of the
 * k_prerotated = 1 comparison path. */
pic_status pic_rope_rotate(const pic_config* cfg, const pic_rope_table* rope, void* x, int32_t n,
                           int32_t num_heads, const int32_t* positions, void* stream);

/* Store new key/value rows in the paged pool (Sec. 3.2.1: keys are cached
 * unrotated).  Row i of k_new/v_new (DEVICE [n][Hkv][D]) goes to slot
 * s = slot_mapping[i] (DEVICE [n]): pool[s/16][h][s%16][:] for every KV head h,
 * pools being DEVICE [num_blocks][Hkv][16][D].  Negative slots are skipped.
 * Slots must be distinct (a repeated slot is a race).  n < 2^24 per call
 * (PIC_EINVAL otherwise).  Bit-exact copy. */
pic_status pic_kv_write(const pic_config* cfg, void* k_pool, void* v_pool, int32_t num_blocks,
                        const void* k_new, const void* v_new, const int32_t* slot_mapping, int32_t n,
                        void* stream);

/* Move whole cache blocks between the pool and another buffer, e.g. to offload
 * them to host memory and bring them back (Sec. 3.2.3, "Native Offloading
 * Compatibility": the blocks hold unrotated keys, so they move between memory
 * tiers with no position bookkeeping and may come back under different block ids
 * and be read at any logical offset).  Block b is the K page run
 * k_pool[b][0..Hkv)[16][D] and the same run of V (Hkv*16*D elements each).
 *  pic_blocks_gather:  dst_k[i] <- k_pool[block_ids[i]], dst_v[i] <- v_pool[block_ids[i]]
 *  pic_blocks_scatter: k_pool[block_ids[i]] <- src_k[i], v_pool[block_ids[i]] <- src_v[i]
 * for i < n.  dst/src are [n][Hkv][16][D] in cfg->dtype, in device memory or in
 * pinned host memory (hipHostMalloc, e.g. a torch tensor created with
 * pin_memory=True); other host memory, managed memory and addresses that are not
 * 16-byte aligned are rejected with PIC_EINVAL.  block_ids is
 * DEVICE [n] and trusted (ids in [0, num_blocks); distinct for a scatter).  One
 * kernel on `stream` copies 16-byte chunks (host buffers are read or written across
 * the host link by the kernel itself); the copies are bit-exact.  n < 2^24 blocks
 * per call (PIC_EINVAL otherwise). */
pic_status pic_blocks_gather(const pic_config* cfg, const void* k_pool, const void* v_pool, int32_t num_blocks,
                             const int32_t* block_ids, int32_t n, void* dst_k, void* dst_v, void* stream);
pic_status pic_blocks_scatter(const pic_config* cfg, void* k_pool, void* v_pool, int32_t num_blocks,
                              const int32_t* block_ids, int32_t n, const void* src_k, const void* src_v,
                              void* stream);

/* Workspace bytes that pic_attn_prefill (is_decode = 0) or pic_attn_decode
 * (is_decode = 1) needs for this configuration and batch: split-KV partial results
 * and, for batches of more than 64 groups (query spans; requests for decode), the
 * work-group table that the call writes there before its attention launch.  May be
 * 0.  Returned through *bytes (the status reports argument errors). */
pic_status pic_workspace_size(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode,
                              size_t* bytes);

/* Prefill attention for the tokens of every PIC_QUERY span.
 *  q  DEVICE [total_q][Hq][D]: one row per query token, request-major, spans and
 *     tokens in sequence order; unrotated unless cfg->k_prerotated.
 *  o  DEVICE [total_q][Hq][D], same order; fully overwritten.
 *  k_pool, v_pool DEVICE [num_blocks][Hkv][16][D] holding every token of every
 *     request (write the call's fresh rows with pic_kv_write first, on the same
 *     stream).
 * Query token t of request r (sequence index n_t) attends to keys j with
 * w(n_t) <= j <= n_t, w being the window start of its span: the span start for
 * PIC_SSEP, 0 for PIC_PDEP, the previous span's window otherwise (0 for the first
 * span).  Keys outside every window are never read. */
pic_status pic_attn_prefill(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                            const pic_rope_table* rope, const void* q, void* o, const void* k_pool,
                            const void* v_pool, int32_t num_blocks, void* workspace, size_t workspace_bytes,
                            void* stream);

/* Decode attention: one query per request, the request's last token n = L_r - 1
 * (already stored with pic_kv_write), with the window of the span holding it.
 *  q, o DEVICE [R][Hq][D]. */
pic_status pic_attn_decode(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                           const pic_rope_table* rope, const void* q, void* o, const void* k_pool,
                           const void* v_pool, int32_t num_blocks, void* workspace, size_t workspace_bytes,
                           void* stream);

/* pic_attn_decode for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments minus the workspace, the same kernels and results.  The split-KV
 * partials and the group table live in a 64 MiB device scratch array inside the
 * library, one per GPU the library runs on, held until the process ends; the call
 * allocates nothing.  A batch needing more scratch than that is refused with
 * PIC_EWORKSPACE before anything is launched (pic_workspace_size(cfg, batch, 1)
 * gives the need).  Every call on one GPU shares that GPU's scratch: calls that
 * overlap on one GPU (concurrent streams, or from several threads) race and must
 * be serialised by the caller.  The stream must belong to the current device. */
pic_status pic_attn_decode_noalloc(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                                   const pic_rope_table* rope, const void* q, void* o, const void* k_pool,
                                   const void* v_pool, int32_t num_blocks, void* stream);

/* Test hook: the work decomposition the prefill/decode call would launch, as
 * rows of 8 int32 {request, kv_head, first query row (flattened token*G+head
 * offset within the span), end query row, key begin, key end, span first token,
 * partial slot or -1}.  Writes min(*n_items, capacity) rows to `items` (HOST)
 * and the full count to *n_items.  No HIP call is made. */
pic_status pic_plan_debug(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode,
                          int32_t* items, int32_t capacity, int32_t* n_items);

/* Test hook: the launch shape of the prefill/decode call (HOST int32 shape[5]):
 * {blocks of the attention launch, blocks of the split-merge launch (0: none),
 *  groups (query spans, or requests for decode), plan-upload launches that write the
 *  group table into the workspace (0 when the groups travel as kernel arguments),
 *  split partial slots}.  Every call is one attention launch and at most one merge
 *  launch, whatever the batch size.  No HIP call is made. */
pic_status pic_plan_shape(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode, int32_t* shape);

#ifdef __cplusplus
}
#endif

#endif /* PIC_ATTN_H */
