// Internal types shared by the host planner (pic_host.cpp) and the HIP kernels
// (pic_kernels.hip).  Not part of the public ABI.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace pic {

constexpr int kBlock = 16;        // tokens per KV block
#ifndef PIC_TILE_ROWS
#define PIC_TILE_ROWS 256
#endif
#ifndef PIC_TILE_KEYS
#define PIC_TILE_KEYS 64
#endif
constexpr int kTileRows = PIC_TILE_ROWS;  // query rows (token x head-in-group) per prefill workgroup
constexpr int kTileKeys = PIC_TILE_KEYS;  // keys per K/V tile of the prefill kernel
constexpr int kMaxGroups = 64;    // groups passed by value as a kernel argument (arguments < 4 KB)
constexpr int kUploadGroups = 80; // groups carried by one plan-upload launch
constexpr int kTargetCUs = 256;   // MI355X compute units the split policy fills
constexpr int kMergeRows = 8;     // rows per block of the split merge
constexpr int kDecTileKeys = 16;  // keys per decode tile (one cache block)
constexpr int kDecMaxG = 64;      // query heads per KV head the decode kernel handles
#ifndef PIC_DEC_HEADS_D128
#define PIC_DEC_HEADS_D128 8
#endif
// Waves of a wide decode workgroup (and K/V head slots of its LDS stages)
constexpr int dec_heads(int head_dim) { return head_dim == 128 ? PIC_DEC_HEADS_D128 : 8; }
// Waves per KV head in the decode kernel: each takes 16 of the KV head's query
// heads (the columns of its 16x16 MFMA tiles)
constexpr int dec_col_blocks(int group) { return group <= 16 ? 1 : group <= 32 ? 2 : 4; }
// Waves (and head slots) of a decode workgroup: the model's KV heads times the
// waves each needs, rounded up to 2 or 4 when that is at most 4 (three 2-wave or
// two 4-wave workgroups share a CU), else the wide workgroup
constexpr int dec_waves(int head_dim, int hkv, int group) {
    return hkv * dec_col_blocks(group) <= 2 ? 2 : hkv * dec_col_blocks(group) <= 4 ? 4 : dec_heads(head_dim);
}
// Decode workgroups of `waves` waves resident on one CU (LDS-bound)
constexpr int dec_wgs_per_cu(int waves) { return waves == 2 ? 3 : waves == 4 ? 2 : 1; }
// KV heads per decode workgroup
constexpr int dec_kv_per_wg(int head_dim, int hkv, int group) {
    return dec_waves(head_dim, hkv, group) / dec_col_blocks(group);
}

// One query span of one request (prefill) or one request's last token (decode).
// Its work items are (row tile, KV head, key split) triples -- (key split, head
// group) for the decode kernel -- enumerated from item_base.  Partial results of
// split groups take consecutive slots from part_base, and their merge blocks
// consecutive block indices of the merge launch from merge_base.  item_base and
// merge_base are non-decreasing over the groups, so with the groups in the kernel
// arguments a block finds its group by binary search.
struct Group {
    int32_t req;         // request index (row of the block table)
    int32_t tok0;        // sequence index of the span's first query token
    int32_t n_tok;       // query tokens in the span
    int32_t q_row0;      // row of tok0 in q / o
    int32_t win;         // window start of the span's tokens
    int32_t pos_off;     // offset of the request's token 0 in `positions`
    int32_t n_rt;        // row tiles (ceil(n_tok * G / kTileRows))
    int32_t n_split;     // key splits per (row tile, KV head)
    int32_t split_keys;  // keys per split (a multiple of kTileKeys)
    int32_t item_base;   // first item (block index) of the group; a multiple of 8 (prefill)
    int32_t part_base;   // first partial slot (split groups)
    int32_t merge_base;  // first block of the merge launch (split groups)
};

// The work of one call: one attention launch of n_items blocks and one merge launch
// of n_merge blocks, whatever the number of groups.  Up to kMaxGroups groups travel
// in g[] (binary-searched by the blocks); a larger batch has its groups in the
// caller's workspace (`table`), written there by plan-upload launches on the same
// stream, with the group index of every attention block in item_map and of every
// merge block in merge_map.
struct Plan {
    int32_t n_groups;
    int32_t n_items;     // blocks of the attention launch
    int32_t n_merge;     // blocks of the merge launch
    int32_t pad_;
    const Group* table;       // device [n_groups], or null when g[] holds the groups
    const int32_t* item_map;  // device [n_items]: group of each attention block
    const int32_t* merge_map; // device [n_merge]: group of each merge block
    Group g[kMaxGroups];
};

// Arguments of one plan-upload launch: groups [first, first + n) of the call, and
// where the block ranges of the chunk's last group end.
struct PlanUpload {
    Group* table;
    int32_t* item_map;
    int32_t* merge_map;
    int32_t first;
    int32_t n;
    int32_t item_end;
    int32_t merge_end;
    Group g[kUploadGroups];
};

// last group whose `field` is <= b (the fields are non-decreasing over groups)
template <int32_t Group::*field>
__host__ __device__ inline int plan_search(const Plan& p, int b) {
    int lo = 0, hi = p.n_groups - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (p.g[mid].*field <= b) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// RoPE phase step of pair i as a 64-bit fraction of a revolution per position,
// round(frac(omega_i / 2pi) * 2^64); 0 for pairs that do not turn
struct RopeSteps {
    uint64_t s[64];
};

struct Args {
    uint64_t fstep[64];       // RopeSteps of the call
    // q and K are read in "kernel layout": its 8-element chunk c is the model's chunk
    // (chunk_map >> 4c) & 15.  Identity except for NeoX pairing with a partial rotary
    // width R, where kernel pair (i, i + D/2) must be the model pair (i, i + R/2) for
    // i < R/2 and a pass-through pair (step 0) otherwise.
    uint64_t chunk_map;
    const void* q;
    void* o;
    const void* k_pool;
    const void* v_pool;
    const int32_t* block_tables;
    const int32_t* positions;
    const float* rope_table;  // [rope_len][D/2] 8-byte entries (format by dtype) or null
    float* part_o;            // [slot][kTileRows][D] split partial outputs: prefill stores
                              // them normalised by the split's sum as bf16, decode
                              // unnormalised as fp32
    float* part_ml;           // [slot][kTileRows][2] running max (log2 units) and sum
    float scale_log2;         // softmax scale * log2(e)
    int32_t max_blocks;
    int32_t rope_len;
    int32_t hq;
    int32_t hkv;
    int32_t group;            // G = hq / hkv
};

// Records msg as the thread's last error (pic_last_error) and returns st.
int32_t host_fail(int32_t st, const char* msg);

// Launchers implemented in pic_kernels.hip.  Each returns a hipError_t value.
int launch_kv_write(int dtype, int hkv, int d, void* k_pool, void* v_pool, const void* k_new,
                    const void* v_new, const int32_t* slots, int n, void* stream);
int launch_rope_table(int dtype, int d, const RopeSteps& steps, int n_pos, float* table, void* stream);
int launch_blocks_copy(int dtype, int hkv, int d, void* k_pool, void* v_pool, void* k_buf, void* v_buf,
                       const int32_t* block_ids, int n, bool to_pool, void* stream);
int launch_rope_rotate(int dtype, int style, int d, int rot_half, const RopeSteps& steps, const float* table, int rope_len, void* x,
                       int n, int heads, const int32_t* positions, void* stream);
int launch_attention(int dtype, int style, int d, bool rope, const Plan& plan, const Args& args, void* stream);
int launch_decode(int style, int d, bool rope, const Plan& plan, const Args& args, void* stream);
int launch_plan_upload(const PlanUpload& up, void* stream);

// Device scratch of the no-allocation entry point: kScratchBytes on each device,
// shared by every call on that device.  scratch_region returns the current
// device's address of it (a hipError_t value).
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
int scratch_region(void** ptr);

}  // namespace pic
