// Host side of libpic_attn: argument validation, the work planner and the
// C-ABI entry points declared in include/pic_attn.h.
//
// The planner turns the host span descriptor into launch groups: one group per
// PIC_QUERY span (prefill) or per request (decode), each with its window start
// (Sec. 3.1.1: SSEP -> span start, PDEP -> 0, unflagged -> previous span's
// window), its row tiles and its key splits.  A call is one attention launch (and
// one merge launch when keys are split) whatever the batch size.  Up to
// kMaxGroups groups travel to the kernels by value as a kernel argument; larger
// batches get their group table written into the caller's workspace by small
// plan-upload launches whose arguments carry the groups.  No call enqueues a
// host-to-device copy.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "pic_attn.h"
#include "pic_internal.h"

namespace {

// both structures travel as kernel arguments
static_assert(sizeof(pic::Plan) + sizeof(pic::Args) <= 4096, "kernel arguments must stay within 4 KB");
static_assert(sizeof(pic::PlanUpload) <= 4096, "kernel arguments must stay within 4 KB");

thread_local std::string g_error;

pic_status fail(pic_status st, const std::string& msg) {
    g_error = msg;
    return st;
}

// The kernels move 16-byte chunks of every tensor (some of them straight into LDS)
// and 4-byte words of the int32 arrays: addresses that do not allow it are refused.
static bool misaligned(const void* p, uintptr_t to) { return p != nullptr && reinterpret_cast<uintptr_t>(p) % to != 0; }

pic_status check_config(const pic_config* c) {
    if (c == nullptr) return fail(PIC_EINVAL, "cfg is NULL");
    if (c->num_q_heads <= 0 || c->num_kv_heads <= 0) return fail(PIC_EINVAL, "head counts must be positive");
    if (c->num_q_heads % c->num_kv_heads != 0) return fail(PIC_EINVAL, "num_q_heads must be a multiple of num_kv_heads");
    if (c->block_size != pic::kBlock) return fail(PIC_EUNSUPPORTED, "block_size must be 16");
    if (c->head_dim != 64 && c->head_dim != 128) return fail(PIC_EUNSUPPORTED, "head_dim must be 64 or 128");
    if (c->dtype != PIC_BF16 && c->dtype != PIC_F32) return fail(PIC_EUNSUPPORTED, "dtype must be PIC_BF16 or PIC_F32");
    if (c->rope_style != PIC_ROPE_NEOX && c->rope_style != PIC_ROPE_GPTJ) return fail(PIC_EINVAL, "unknown rope_style");
    if (!(c->rope_theta > 0.0) || !std::isfinite(c->rope_theta)) return fail(PIC_EINVAL, "rope_theta must be positive");
    if (!(c->softmax_scale >= 0.f) || !std::isfinite(c->softmax_scale)) return fail(PIC_EINVAL, "softmax_scale must be >= 0");
    if (c->k_prerotated != 0 && c->k_prerotated != 1) return fail(PIC_EINVAL, "k_prerotated must be 0 or 1");
    const int rd = c->rotary_dim ? c->rotary_dim : c->head_dim;
    if (rd < 2 || rd > c->head_dim || rd % 2) return fail(PIC_EINVAL, "rotary_dim must be 0 or even in [2, head_dim]");
    if (rd < c->head_dim && c->rope_style == PIC_ROPE_NEOX && rd % 16 != 0)
        return fail(PIC_EUNSUPPORTED, "partial rotary_dim with NeoX pairing must be a multiple of 16");
    if (c->inv_freq)
        for (int i = 0; i < rd / 2; ++i)
            if (!std::isfinite(c->inv_freq[i])) return fail(PIC_EINVAL, "inv_freq must be finite");
    return PIC_OK;
}

// Window start of every span of request r (the rule of the span flags, or the
// explicit override).
pic_status span_windows(const pic_batch_host* b, int r, std::vector<int32_t>& w) {
    const int s0 = b->cu_spans[r], s1 = b->cu_spans[r + 1];
    w.assign(s1 - s0, 0);
    int32_t prev = 0;
    for (int k = s0; k < s1; ++k) {
        const int32_t f = b->span_flags[k];
        int32_t wk;
        if (b->span_window != nullptr && b->span_window[k] >= 0)
            wk = b->span_window[k];
        else if (f & PIC_SSEP)
            wk = b->span_start[k];
        else if (f & PIC_PDEP)
            wk = 0;
        else
            wk = prev;
        w[k - s0] = wk;
        prev = wk;
    }
    return PIC_OK;
}

pic_status check_batch(const pic_batch_host* b) {
    if (b == nullptr) return fail(PIC_EINVAL, "batch is NULL");
    if (b->num_reqs < 0) return fail(PIC_EINVAL, "num_reqs < 0");
    if (b->num_reqs == 0) return PIC_OK;
    if (!b->seq_lens || !b->cu_spans || !b->span_start || !b->span_flags)
        return fail(PIC_EINVAL, "batch arrays must not be NULL");
    if (b->cu_spans[0] != 0) return fail(PIC_EINVAL, "cu_spans[0] must be 0");
    int64_t total = 0;
    for (int r = 0; r < b->num_reqs; ++r) {
        const int32_t L = b->seq_lens[r];
        if (L < 1) return fail(PIC_EINVAL, "seq_lens[" + std::to_string(r) + "] must be >= 1");
        total += L;
        const int s0 = b->cu_spans[r], s1 = b->cu_spans[r + 1];
        if (s1 <= s0) return fail(PIC_EINVAL, "request " + std::to_string(r) + " has no span");
        if (b->span_start[s0] != 0) return fail(PIC_EINVAL, "first span of a request must start at 0");
        for (int k = s0; k < s1; ++k) {
            const int32_t f = b->span_flags[k];
            if (f & ~(PIC_SSEP | PIC_PDEP | PIC_QUERY)) return fail(PIC_EINVAL, "unknown span flag bits");
            if ((f & PIC_SSEP) && (f & PIC_PDEP)) return fail(PIC_EINVAL, "a span cannot be both SSEP and PDEP");
            if (b->span_start[k] < 0 || b->span_start[k] >= L) return fail(PIC_EINVAL, "span_start out of range");
            if (k > s0 && b->span_start[k] <= b->span_start[k - 1])
                return fail(PIC_EINVAL, "span_start must be strictly increasing within a request");
            if (b->span_window != nullptr && b->span_window[k] >= 0 && b->span_window[k] > b->span_start[k])
                return fail(PIC_EINVAL, "span_window must not exceed the span start");
        }
    }
    if (total > INT32_MAX) return fail(PIC_EINVAL, "total tokens exceed int32");
    return PIC_OK;
}

struct HostPlan {
    std::vector<pic::Group> groups;
    int64_t n_items = 0;       // blocks of the attention launch
    int64_t n_parts = 0;       // split partial slots
    int64_t n_merge = 0;       // blocks of the merge launch
    bool dec_kernel = false;   // decode through the one-query kernel (bf16, G <= kDecMaxG)
};

int32_t round_up(int64_t x, int64_t m) { return (int32_t)((x + m - 1) / m * m); }

// Decode workgroups per (request, key split): KV heads in groups of dec_kv_per_wg.
int64_t dec_head_groups(const pic_config* c) {
    const int64_t per_wg = pic::dec_kv_per_wg(c->head_dim, c->num_kv_heads, c->num_q_heads / c->num_kv_heads);
    return (c->num_kv_heads + per_wg - 1) / per_wg;
}

// Groups, their split policy and bases.  f32 groups hold one item per
// (query token, query head); bf16 groups hold (row tile, KV head, split) items.
pic_status make_plan(const pic_config* c, const pic_batch_host* b, bool decode, HostPlan& hp) {
    hp.groups.clear();
    hp.n_parts = 0;
    const int G = c->num_q_heads / c->num_kv_heads;
    std::vector<int32_t> w;
    int64_t pos_off = 0, q_row = 0;
    for (int r = 0; r < b->num_reqs; ++r) {
        span_windows(b, r, w);
        const int s0 = b->cu_spans[r], s1 = b->cu_spans[r + 1];
        const int32_t L = b->seq_lens[r];
        if (decode) {
            pic::Group g{};
            g.req = r;
            g.tok0 = L - 1;
            g.n_tok = 1;
            g.q_row0 = r;
            g.win = w[s1 - s0 - 1];
            g.pos_off = (int32_t)pos_off;
            hp.groups.push_back(g);
        } else {
            for (int k = s0; k < s1; ++k) {
                if (!(b->span_flags[k] & PIC_QUERY)) continue;
                const int32_t e = k + 1 < s1 ? b->span_start[k + 1] : L;
                pic::Group g{};
                g.req = r;
                g.tok0 = b->span_start[k];
                g.n_tok = e - g.tok0;
                g.q_row0 = (int32_t)q_row;
                g.win = w[k - s0];
                g.pos_off = (int32_t)pos_off;
                q_row += g.n_tok;
                hp.groups.push_back(g);
            }
        }
        pos_off += L;
    }
    if (q_row > INT32_MAX / 2) return fail(PIC_EINVAL, "too many query rows");

    hp.dec_kernel = decode && c->dtype == PIC_BF16 && G <= pic::kDecMaxG;
    if (hp.dec_kernel) {
        // Decode items are (request, key split, group of KV heads).  A wide workgroup
        // holds a CU (narrow ones share it three or two ways), so cut the keys into
        // chunks of about the average work per resident workgroup (at least 4 cache
        // blocks) and balance the splits of each request.
        const int64_t n_hg = dec_head_groups(c);
        int64_t tiles_total = 0;
        for (auto& g : hp.groups)
            tiles_total += n_hg * (((int64_t)g.tok0 + 1 - g.win + pic::kDecTileKeys - 1) / pic::kDecTileKeys);
        const int64_t target = (int64_t)pic::kTargetCUs * pic::dec_wgs_per_cu(pic::dec_waves(c->head_dim, c->num_kv_heads, G));
        const int64_t chunk = std::max<int64_t>(4, (tiles_total + target - 1) / target);
        for (auto& g : hp.groups) {
            const int64_t tiles = ((int64_t)g.tok0 + 1 - g.win + pic::kDecTileKeys - 1) / pic::kDecTileKeys;
            g.n_rt = 1;
            g.n_split = (int32_t)((tiles + chunk - 1) / chunk);
            g.split_keys = (int32_t)(((tiles + g.n_split - 1) / g.n_split) * pic::kDecTileKeys);
        }
        std::stable_sort(hp.groups.begin(), hp.groups.end(), [](const pic::Group& x, const pic::Group& y) {
            return std::min<int64_t>(x.split_keys, x.tok0 + 1 - x.win) > std::min<int64_t>(y.split_keys, y.tok0 + 1 - y.win);
        });
    } else if (c->dtype == PIC_F32) {
        for (auto& g : hp.groups) {
            g.n_rt = g.n_tok;
            g.n_split = 1;
            g.split_keys = 0;
        }
    } else {
        // Key splits, counted in 64-key tiles.  Split when the unsplit items cannot
        // fill the chip (chunks of the average work per CU), or when some item is
        // much longer than the average work per CU, which would leave its CU running
        // alone at the end (chunks of a third of that average).
        int64_t base = 0, tiles_total = 0, max_item = 0;
        for (auto& g : hp.groups) {
            g.n_rt = (int32_t)(((int64_t)g.n_tok * G + pic::kTileRows - 1) / pic::kTileRows);
            const int64_t tiles = ((int64_t)g.tok0 + g.n_tok - g.win + pic::kTileKeys - 1) / pic::kTileKeys;
            base += (int64_t)g.n_rt * c->num_kv_heads;
            tiles_total += (int64_t)g.n_rt * c->num_kv_heads * tiles;
            max_item = std::max(max_item, tiles);
        }
        const double avg = (double)tiles_total / pic::kTargetCUs;
        int64_t cap = INT32_MAX;
        if (base < pic::kTargetCUs)
            cap = std::max<int64_t>(4, (int64_t)std::ceil(avg));
        else if ((double)max_item > 1.25 * avg)
            cap = std::max<int64_t>(32, (int64_t)std::ceil(avg / 3.0));
        for (auto& g : hp.groups) {
            const int64_t tiles = ((int64_t)g.tok0 + g.n_tok - g.win + pic::kTileKeys - 1) / pic::kTileKeys;
            g.n_split = (int32_t)((tiles + cap - 1) / cap);
            g.split_keys = (int32_t)(((tiles + g.n_split - 1) / g.n_split) * pic::kTileKeys);
        }
        // heaviest items first
        std::stable_sort(hp.groups.begin(), hp.groups.end(), [](const pic::Group& x, const pic::Group& y) {
            const int64_t cx = (int64_t)std::min(x.n_tok, pic::kTileRows) * std::min<int64_t>(x.split_keys, x.tok0 + x.n_tok - x.win);
            const int64_t cy = (int64_t)std::min(y.n_tok, pic::kTileRows) * std::min<int64_t>(y.split_keys, y.tok0 + y.n_tok - y.win);
            return cx > cy;
        });
    }
    return PIC_OK;
}

int64_t items_of(const pic_config* c, const HostPlan& hp, const pic::Group& g) {
    if (hp.dec_kernel) return (int64_t)g.n_split * dec_head_groups(c);
    if (c->dtype == PIC_F32) return (int64_t)g.n_tok * c->num_q_heads;
    return (int64_t)g.n_rt * c->num_kv_heads * g.n_split;
}

// Assign every group its item, partial-slot and merge-block bases (one attention
// launch and one merge launch for the whole call) and count the blocks.
pic_status assign_bases(const pic_config* c, HostPlan& hp) {
    int64_t item = 0, part = 0, merge = 0;
    for (auto& g : hp.groups) {
        const int64_t n = items_of(c, hp, g);
        const int64_t n_pad = hp.dec_kernel ? n : round_up(n, 8);
        g.item_base = (int32_t)item;
        g.part_base = (int32_t)part;
        g.merge_base = (int32_t)merge;
        item += n_pad;
        if (hp.dec_kernel) {
            if (g.n_split > 1) {
                part += n;
                merge += (c->num_q_heads + pic::kMergeRows - 1) / pic::kMergeRows;
            }
        } else if (c->dtype != PIC_F32 && g.n_split > 1) {
            part += (int64_t)g.n_rt * c->num_kv_heads * g.n_split;
            merge += (int64_t)g.n_rt * c->num_kv_heads * (pic::kTileRows / pic::kMergeRows);
        }
        // a launch's lanes (blocks x threads) must stay below 2^31
        if (item > (1 << 22) || merge > (1 << 23) || part > (1 << 24))
            return fail(PIC_EINVAL, "batch too large for one call (split it into several calls)");
    }
    hp.n_items = item;
    hp.n_parts = part;
    hp.n_merge = merge;
    return PIC_OK;
}

constexpr size_t kWsAlign = 256;
size_t align_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

// Workspace layout: split partial outputs [n_parts][kTileRows][D] (sized for fp32),
// their (max, sum) pairs [n_parts][kTileRows][2], and -- for batches of more than
// kMaxGroups groups -- the group table with the block -> group maps.
struct WsLayout {
    size_t ml = 0, table = 0, item_map = 0, merge_map = 0, total = 0;
};

WsLayout ws_layout(const pic_config* c, const HostPlan& hp) {
    WsLayout w;
    const size_t parts = (size_t)hp.n_parts * pic::kTileRows;
    w.ml = parts * c->head_dim * sizeof(float);
    w.total = w.ml + parts * 2 * sizeof(float);
    if (hp.groups.size() > (size_t)pic::kMaxGroups) {
        w.table = align_up(w.total);
        w.item_map = align_up(w.table + hp.groups.size() * sizeof(pic::Group));
        w.merge_map = align_up(w.item_map + (size_t)hp.n_items * sizeof(int32_t));
        w.total = w.merge_map + (size_t)hp.n_merge * sizeof(int32_t);
    }
    return w;
}

// The plan of a call: groups with their split policy, then their bases.
pic_status build_plan(const pic_config* c, const pic_batch_host* b, bool decode, HostPlan& hp) {
    pic_status st = make_plan(c, b, decode, hp);
    if (st) return st;
    return assign_bases(c, hp);
}

// Phase step of RoPE pair i: omega_i / 2pi revolutions per position as a 64-bit
// binary fraction, in long double so that the rounding of omega_i stays far below
// the 2^-64 step.  omega_i = theta^(-2i/R) or the given inv_freq[i] for i < R/2,
// nothing past the rotary width.
void phase_steps(const pic_config* c, uint64_t* out) {
    const long double two_pi = 6.283185307179586476925286766559L;
    const int rd = c->rotary_dim ? c->rotary_dim : c->head_dim;
    for (int i = 0; i < c->head_dim / 2; ++i) {
        out[i] = 0;
        if (i >= rd / 2) continue;
        const long double om = c->inv_freq ? (long double)c->inv_freq[i]
                                           : powl((long double)c->rope_theta, -2.0L * i / rd);
        long double rev = om / two_pi;
        rev -= floorl(rev);
        out[i] = (uint64_t)(rev * 18446744073709551616.0L);
    }
}

// Kernel-layout chunk c of q and K (8 elements) -> model chunk, 4 bits per chunk.
// NeoX with rotary width R < D: kernel chunks [0, R/16) and [D/16, D/16 + R/16) are
// the model's two rotary halves, the other kernel chunks the model's pass-through
// chunks [R/8, D/8) in order.
uint64_t chunk_map(const pic_config* c) {
    const int ch = c->head_dim / 8, rd = c->rotary_dim ? c->rotary_dim : c->head_dim;
    int map[16];
    for (int i = 0; i < ch; ++i) map[i] = i;
    if (c->rope_style == PIC_ROPE_NEOX && rd < c->head_dim && !c->k_prerotated) {
        const int rc = rd / 16;
        int next = 2 * rc;
        for (int i = 0; i < ch / 2; ++i) {
            if (i < rc) {
                map[i] = i;
                map[i + ch / 2] = rc + i;
            } else {
                map[i] = next++;
                map[i + ch / 2] = next++;
            }
        }
    }
    uint64_t m = 0;
    for (int i = 0; i < ch; ++i) m |= (uint64_t)map[i] << (4 * i);
    return m;
}

pic_status hip_status(int e, const char* what) {
    if (e != hipSuccess) return fail(PIC_EHIP, std::string(what) + ": " + hipGetErrorString((hipError_t)e));
    return PIC_OK;
}

pic_status run_attention(const pic_config* c, const pic_batch_host* b, const pic_batch_dev* dv,
                         const pic_rope_table* rope, const void* q, void* o, const void* k_pool, const void* v_pool,
                         int32_t num_blocks, void* ws, size_t ws_bytes, void* stream, bool decode) {
    pic_status st = check_config(c);
    if (st) return st;
    if ((st = check_batch(b))) return st;
    if (b->num_reqs == 0) return PIC_OK;
    if (dv == nullptr || dv->block_tables == nullptr || dv->positions == nullptr)
        return fail(PIC_EINVAL, "device batch arrays must not be NULL");
    if (num_blocks <= 0) return fail(PIC_EINVAL, "num_blocks must be positive");
    for (int r = 0; r < b->num_reqs; ++r)
        if ((int64_t)dv->max_blocks * pic::kBlock < b->seq_lens[r])
            return fail(PIC_EINVAL, "max_blocks too small for seq_lens[" + std::to_string(r) + "]");
    if (!k_pool || !v_pool) return fail(PIC_EINVAL, "pools must not be NULL");
    if (rope != nullptr && rope->data != nullptr && rope->len < 0) return fail(PIC_EINVAL, "rope table len < 0");
    if (misaligned(q, 16) || misaligned(o, 16) || misaligned(k_pool, 16) || misaligned(v_pool, 16) ||
        misaligned(ws, 16) || (rope != nullptr && misaligned(rope->data, 16)))
        return fail(PIC_EINVAL, "q, o, the pools, the workspace and the rope table must be 16-byte aligned");
    if (misaligned(dv->block_tables, 4) || misaligned(dv->positions, 4))
        return fail(PIC_EINVAL, "block tables and positions must be 4-byte aligned");

    HostPlan hp;
    if ((st = build_plan(c, b, decode, hp))) return st;
    int64_t rows = 0;
    for (auto& g : hp.groups) rows += g.n_tok;
    if (rows == 0) return PIC_OK;
    if (!q || !o) return fail(PIC_EINVAL, "q and o must not be NULL");
    const WsLayout wl = ws_layout(c, hp);
    if (wl.total > 0 && (ws == nullptr || ws_bytes < wl.total))
        return fail(PIC_EWORKSPACE, "workspace needs " + std::to_string(wl.total) + " bytes");

    pic::Args a{};
    phase_steps(c, a.fstep);
    a.chunk_map = chunk_map(c);
    a.q = q;
    a.o = o;
    a.k_pool = k_pool;
    a.v_pool = v_pool;
    a.block_tables = dv->block_tables;
    a.positions = dv->positions;
    const bool table = rope != nullptr && rope->data != nullptr && rope->len > 0;
    a.rope_table = table ? static_cast<const float*>(rope->data) : nullptr;
    a.rope_len = table ? rope->len : 0;
    char* wsb = static_cast<char*>(ws);
    a.part_o = hp.n_parts ? reinterpret_cast<float*>(wsb) : nullptr;
    a.part_ml = hp.n_parts ? reinterpret_cast<float*>(wsb + wl.ml) : nullptr;
    const double scale = c->softmax_scale > 0.f ? (double)c->softmax_scale : 1.0 / std::sqrt((double)c->head_dim);
    a.scale_log2 = (float)(scale * 1.4426950408889634);
    a.max_blocks = dv->max_blocks;
    a.hq = c->num_q_heads;
    a.hkv = c->num_kv_heads;
    a.group = c->num_q_heads / c->num_kv_heads;

    pic::Plan p;
    std::memset(&p, 0, sizeof(p));
    p.n_groups = (int32_t)hp.groups.size();
    p.n_items = (int32_t)hp.n_items;
    p.n_merge = (int32_t)hp.n_merge;
    if (hp.groups.size() <= (size_t)pic::kMaxGroups) {
        std::copy(hp.groups.begin(), hp.groups.end(), p.g);
    } else {
        // the group table and block maps go to the workspace, written on the stream
        // ahead of the attention launch by plan-upload launches of up to
        // kUploadGroups groups each (their arguments carry the groups)
        pic::Group* tab = reinterpret_cast<pic::Group*>(wsb + wl.table);
        int32_t* imap = reinterpret_cast<int32_t*>(wsb + wl.item_map);
        int32_t* mmap = reinterpret_cast<int32_t*>(wsb + wl.merge_map);
        p.table = tab;
        p.item_map = imap;
        p.merge_map = mmap;
        const size_t n = hp.groups.size();
        for (size_t first = 0; first < n; first += pic::kUploadGroups) {
            pic::PlanUpload u;
            std::memset(&u, 0, sizeof(u));
            u.table = tab;
            u.item_map = imap;
            u.merge_map = mmap;
            u.first = (int32_t)first;
            u.n = (int32_t)std::min<size_t>(pic::kUploadGroups, n - first);
            std::copy(hp.groups.begin() + first, hp.groups.begin() + first + u.n, u.g);
            const bool last = first + u.n == n;
            u.item_end = last ? (int32_t)hp.n_items : hp.groups[first + u.n].item_base;
            u.merge_end = last ? (int32_t)hp.n_merge : hp.groups[first + u.n].merge_base;
            if ((st = hip_status(pic::launch_plan_upload(u, stream), "plan upload launch"))) return st;
        }
    }
    const bool rope_on = c->k_prerotated == 0;
    const int e = hp.dec_kernel ? pic::launch_decode(c->rope_style, c->head_dim, rope_on, p, a, stream)
                                : pic::launch_attention(c->dtype, c->rope_style, c->head_dim, rope_on, p, a, stream);
    return hip_status(e, "attention launch");
}

}  // namespace

namespace pic {
pic_status host_fail(pic_status st, const char* msg) { return fail(st, msg); }
}  // namespace pic

extern "C" {

int32_t pic_version(void) { return 100; }

const char* pic_last_error(void) { return g_error.c_str(); }

pic_status pic_rope_table_bytes(const pic_config* cfg, int32_t num_positions, size_t* bytes) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if (num_positions < 0 || bytes == nullptr) return fail(PIC_EINVAL, "bad num_positions or bytes pointer");
    // float32 tables hold (cos, sin) as two floats, bf16 tables as one bf16 pair
    *bytes = (size_t)num_positions * (cfg->head_dim / 2) * (cfg->dtype == PIC_F32 ? 8 : 4);
    return PIC_OK;
}

pic_status pic_rope_table_build(const pic_config* cfg, int32_t num_positions, void* table, void* stream) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if (num_positions < 0) return fail(PIC_EINVAL, "num_positions < 0");
    if (num_positions > 0 && table == nullptr) return fail(PIC_EINVAL, "table is NULL");
    if (misaligned(table, 16)) return fail(PIC_EINVAL, "table must be 16-byte aligned");
    pic::RopeSteps steps;
    phase_steps(cfg, steps.s);
    return hip_status(pic::launch_rope_table(cfg->dtype, cfg->head_dim, steps, num_positions,
                                             static_cast<float*>(table), stream),
                      "rope table launch");
}

pic_status pic_rope_rotate(const pic_config* cfg, const pic_rope_table* rope, void* x, int32_t n, int32_t num_heads,
                           const int32_t* positions, void* stream) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if (n < 0 || num_heads <= 0) return fail(PIC_EINVAL, "bad n or num_heads");
    if (n == 0) return PIC_OK;
    if (x == nullptr || positions == nullptr) return fail(PIC_EINVAL, "x and positions must not be NULL");
    if (misaligned(x, 16) || misaligned(positions, 4) || (rope != nullptr && misaligned(rope->data, 16)))
        return fail(PIC_EINVAL, "x and the rope table must be 16-byte aligned, positions 4-byte aligned");
    const bool table = rope != nullptr && rope->data != nullptr && rope->len > 0;
    pic::RopeSteps steps;
    phase_steps(cfg, steps.s);
    const int rot_half = (cfg->rotary_dim ? cfg->rotary_dim : cfg->head_dim) / 2;
    return hip_status(pic::launch_rope_rotate(cfg->dtype, cfg->rope_style, cfg->head_dim, rot_half, steps,
                                              table ? static_cast<const float*>(rope->data) : nullptr,
                                              table ? rope->len : 0, x, n, num_heads, positions, stream),
                      "rope rotate launch");
}

pic_status pic_kv_write(const pic_config* cfg, void* k_pool, void* v_pool, int32_t num_blocks, const void* k_new,
                        const void* v_new, const int32_t* slot_mapping, int32_t n, void* stream) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if (n < 0 || num_blocks < 0) return fail(PIC_EINVAL, "n and num_blocks must be >= 0");
    if (n == 0) return PIC_OK;
    if (!k_pool || !v_pool || !k_new || !v_new || !slot_mapping) return fail(PIC_EINVAL, "NULL buffer");
    if (num_blocks == 0) return fail(PIC_EINVAL, "empty pool");
    if (misaligned(k_pool, 16) || misaligned(v_pool, 16) || misaligned(k_new, 16) || misaligned(v_new, 16) ||
        misaligned(slot_mapping, 4))
        return fail(PIC_EINVAL, "pools and new rows must be 16-byte aligned, slot_mapping 4-byte aligned");
    // one workgroup of up to 256 lanes per row: the grid's lane count must stay below 2^32
    if (n >= (1 << 24)) return fail(PIC_EINVAL, "n must be < 2^24 rows per call");
    return hip_status(pic::launch_kv_write(cfg->dtype, cfg->num_kv_heads, cfg->head_dim, k_pool, v_pool, k_new, v_new,
                                           slot_mapping, n, stream),
                      "kv_write launch");
}

// A pointer the kernels can dereference: device memory as it is, pinned host memory
// (hipHostMalloc) through its device mapping.  Anything else -- pageable host memory,
// managed memory -- is rejected, since a kernel touching it could fault.
static pic_status kernel_view(const void* p, const char* what, void** out) {
    hipPointerAttribute_t at{};
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(PIC_EINVAL, std::string(what) + " is neither device memory nor pinned host memory");
    }
    if (at.type == hipMemoryTypeDevice) {
        *out = const_cast<void*>(p);
        return PIC_OK;
    }
    unsigned int flags = 0;
    if (at.type == hipMemoryTypeHost && at.devicePointer != nullptr &&
        hipHostGetFlags(&flags, const_cast<void*>(p)) == hipSuccess) {
        *out = at.devicePointer;
        return PIC_OK;
    }
    (void)hipGetLastError();
    return fail(PIC_EINVAL, std::string(what) + " is neither device memory nor pinned host memory");
}

static pic_status blocks_copy(const pic_config* cfg, void* k_pool, void* v_pool, int32_t num_blocks,
                              const int32_t* block_ids, int32_t n, void* k_buf, void* v_buf, bool to_pool,
                              void* stream) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if (n < 0 || num_blocks < 0) return fail(PIC_EINVAL, "n and num_blocks must be >= 0");
    if (n == 0) return PIC_OK;
    if (!k_pool || !v_pool || !k_buf || !v_buf || !block_ids) return fail(PIC_EINVAL, "NULL buffer");
    if (num_blocks == 0) return fail(PIC_EINVAL, "empty pool");
    // one workgroup of 256 lanes per block: the grid's lane count must stay below 2^32
    if (n >= (1 << 24)) return fail(PIC_EINVAL, "n must be < 2^24 blocks per call");
    void *kb = nullptr, *vb = nullptr;
    if ((st = kernel_view(k_buf, to_pool ? "src_k" : "dst_k", &kb))) return st;
    if ((st = kernel_view(v_buf, to_pool ? "src_v" : "dst_v", &vb))) return st;
    // the kernel moves 16-byte chunks
    for (const void* p : {(const void*)k_pool, (const void*)v_pool, (const void*)kb, (const void*)vb})
        if (reinterpret_cast<uintptr_t>(p) % 16) return fail(PIC_EINVAL, "pool and buffer addresses must be 16-byte aligned");
    return hip_status(pic::launch_blocks_copy(cfg->dtype, cfg->num_kv_heads, cfg->head_dim, k_pool, v_pool, kb, vb,
                                              block_ids, n, to_pool, stream),
                      "blocks_copy launch");
}

pic_status pic_blocks_gather(const pic_config* cfg, const void* k_pool, const void* v_pool, int32_t num_blocks,
                             const int32_t* block_ids, int32_t n, void* dst_k, void* dst_v, void* stream) {
    return blocks_copy(cfg, const_cast<void*>(k_pool), const_cast<void*>(v_pool), num_blocks, block_ids, n, dst_k,
                       dst_v, false, stream);
}

pic_status pic_blocks_scatter(const pic_config* cfg, void* k_pool, void* v_pool, int32_t num_blocks,
                              const int32_t* block_ids, int32_t n, const void* src_k, const void* src_v,
                              void* stream) {
    return blocks_copy(cfg, k_pool, v_pool, num_blocks, block_ids, n, const_cast<void*>(src_k),
                       const_cast<void*>(src_v), true, stream);
}

pic_status pic_workspace_size(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode, size_t* bytes) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if ((st = check_batch(batch))) return st;
    if (bytes == nullptr) return fail(PIC_EINVAL, "bytes is NULL");
    HostPlan hp;
    if ((st = build_plan(cfg, batch, is_decode != 0, hp))) return st;
    *bytes = ws_layout(cfg, hp).total;
    return PIC_OK;
}

pic_status pic_attn_prefill(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                            const pic_rope_table* rope, const void* q, void* o, const void* k_pool, const void* v_pool,
                            int32_t num_blocks, void* workspace, size_t workspace_bytes, void* stream) {
    return run_attention(cfg, batch, dev, rope, q, o, k_pool, v_pool, num_blocks, workspace, workspace_bytes, stream,
                         false);
}

pic_status pic_attn_decode(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                           const pic_rope_table* rope, const void* q, void* o, const void* k_pool, const void* v_pool,
                           int32_t num_blocks, void* workspace, size_t workspace_bytes, void* stream) {
    return run_attention(cfg, batch, dev, rope, q, o, k_pool, v_pool, num_blocks, workspace, workspace_bytes, stream,
                         true);
}

pic_status pic_attn_decode_noalloc(const pic_config* cfg, const pic_batch_host* batch, const pic_batch_dev* dev,
                                   const pic_rope_table* rope, const void* q, void* o, const void* k_pool,
                                   const void* v_pool, int32_t num_blocks, void* stream) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if ((st = check_batch(batch))) return st;
    HostPlan hp;
    if ((st = build_plan(cfg, batch, true, hp))) return st;
    const size_t need = ws_layout(cfg, hp).total;
    if (need > pic::kScratchBytes)
        return fail(PIC_EWORKSPACE, "batch needs " + std::to_string(need) + " bytes of scratch; the no-allocation "
                    "entry point has " + std::to_string(pic::kScratchBytes) + " (use pic_attn_decode with a workspace)");
    void* ws = nullptr;
    if ((st = hip_status(pic::scratch_region(&ws), "scratch address"))) return st;
    return run_attention(cfg, batch, dev, rope, q, o, k_pool, v_pool, num_blocks, ws, pic::kScratchBytes, stream,
                         true);
}

pic_status pic_plan_debug(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode, int32_t* items,
                          int32_t capacity, int32_t* n_items) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if ((st = check_batch(batch))) return st;
    if (n_items == nullptr || capacity < 0 || (capacity > 0 && items == nullptr))
        return fail(PIC_EINVAL, "bad output arguments");
    HostPlan hp;
    if ((st = build_plan(cfg, batch, is_decode != 0, hp))) return st;
    const int G = cfg->num_q_heads / cfg->num_kv_heads;
    int64_t n = 0;
    auto emit = [&](int32_t r, int32_t h, int32_t rl, int32_t rh, int32_t kl, int32_t kh, int32_t t0, int32_t slot) {
        if (n < capacity) {
            int32_t* it = items + n * 8;
            it[0] = r; it[1] = h; it[2] = rl; it[3] = rh; it[4] = kl; it[5] = kh; it[6] = t0; it[7] = slot;
        }
        ++n;
    };
    {
        for (size_t gi = 0; gi < hp.groups.size(); ++gi) {
            const pic::Group& g = hp.groups[gi];
            if (hp.dec_kernel) {
                const int64_t n_hg = dec_head_groups(cfg);
                for (int s = 0; s < g.n_split; ++s) {
                    const int32_t kl = g.win + s * g.split_keys;
                    const int32_t kh = std::min(kl + g.split_keys, g.tok0 + 1);
                    if (kl >= kh) continue;
                    for (int kvh = 0; kvh < cfg->num_kv_heads; ++kvh) {
                        const int32_t slot =
                            g.n_split > 1 ? (int32_t)(g.part_base + s * n_hg + kvh / pic::dec_kv_per_wg(cfg->head_dim, cfg->num_kv_heads, G)) : -1;
                        emit(g.req, kvh, 0, G, kl, kh, g.tok0, slot);
                    }
                }
                continue;
            }
            if (cfg->dtype == PIC_F32) {
                for (int t = 0; t < g.n_tok; ++t)
                    for (int h = 0; h < cfg->num_q_heads; ++h) {
                        const int32_t row = t * G + h % G;
                        emit(g.req, h / G, row, row + 1, g.win, g.tok0 + t + 1, g.tok0, -1);
                    }
                continue;
            }
            for (int kvh = 0; kvh < cfg->num_kv_heads; ++kvh)
                for (int s = 0; s < g.n_split; ++s)
                    for (int rt = 0; rt < g.n_rt; ++rt) {
                        const int32_t rl = rt * pic::kTileRows;
                        const int32_t rh = std::min(rl + pic::kTileRows, g.n_tok * G);
                        const int32_t t_last = g.tok0 + (rh - 1) / G;
                        const int32_t kl = g.win + s * g.split_keys;
                        const int32_t kh = std::min(kl + g.split_keys, t_last + 1);
                        if (kl >= kh) continue;
                        const int32_t slot =
                            g.n_split > 1 ? g.part_base + (kvh * g.n_split + s) * g.n_rt + rt : -1;
                        emit(g.req, kvh, rl, rh, kl, kh, g.tok0, slot);
                    }
        }
    }
    *n_items = (int32_t)std::min<int64_t>(n, INT32_MAX);
    return PIC_OK;
}

pic_status pic_plan_shape(const pic_config* cfg, const pic_batch_host* batch, int32_t is_decode, int32_t* shape) {
    pic_status st = check_config(cfg);
    if (st) return st;
    if ((st = check_batch(batch))) return st;
    if (shape == nullptr) return fail(PIC_EINVAL, "shape is NULL");
    HostPlan hp;
    if ((st = build_plan(cfg, batch, is_decode != 0, hp))) return st;
    const int64_t n = (int64_t)hp.groups.size();
    shape[0] = (int32_t)hp.n_items;
    shape[1] = (int32_t)hp.n_merge;
    shape[2] = (int32_t)n;
    shape[3] = n > pic::kMaxGroups ? (int32_t)((n + pic::kUploadGroups - 1) / pic::kUploadGroups) : 0;
    shape[4] = (int32_t)hp.n_parts;
    return PIC_OK;
}

}  // extern "C"
