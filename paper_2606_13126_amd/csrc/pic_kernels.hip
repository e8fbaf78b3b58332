// HIP kernels of libpic_attn for MI355X (gfx950, CDNA4).
//
//  * kv_write      scatter of unrotated K/V rows into the paged pool (Sec. 3.2.1:
//                  the cache keeps keys without positional rotation).
//  * rope_table    the cos/sin lookup table of Sec. 3.2.2, built in float64.
//  * rope_rotate   conventional in-place rotary embedding (comparison path only).
//  * prefill_bf16  paged flash attention, bf16 MFMA (v_mfma_f32_32x32x16_bf16) for
//                  S^T = K Q^T and O^T = V^T P^T, RoPE fused into the K-tile load
//                  (Sec. 3.2.2: load tile, look up cos/sin at the tile's positions,
//                  rotate, then the dot products), exp2 online softmax, window mask
//                  of Sec. 3.1.1 with whole-block skipping, optional key splits.
//  * merge         combines key-split partial results (log-sum-exp merge).
//  * attn_f32      fp32 VALU flash attention for the float32 path.
//
// Layouts: pools [num_blocks][Hkv][16][D]; q/o [rows][Hq][D]; positions int32 per
// token, request-major.  One workgroup of the bf16 kernel owns up to 256 query rows
// (token x query head of one KV head's group) and one key range.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "pic_internal.h"

namespace pic {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr int kNeox = 0;
constexpr float kNegBig = -1.0e30f;  // finite "minus infinity" for running maxima

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// (a.lo * b.lo + a.hi * b.hi) of two bf16 pairs, fp32 result.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), 0.0f,
                                           false);
}

// ---------------------------------------------------------------------------------
// K rotation blocks.  A pair (x, y) turns into (x c - y s, y c + x s) as two
// 2-element dot products with the table entry e = (c, s): (x, y).(c, -s), the sign
// applied by the instruction's neg_hi modifier, and (y, x).(c, s).  The builtin
// dot product with a zero addend compiles to a v_mov of zero plus the accumulating
// VOP2 form (which has no modifiers); these blocks issue the VOP3P form with an
// inline-constant zero addend.  A DOT result read by another VALU instruction needs
// 3 wait states on gfx950, which the compiler cannot see inside inline assembly:
// each block orders its eight dot products before the four conversions that read
// them, so every result is read at least three instructions after it is written and
// no s_nop is needed.  Nothing outside a block reads a DOT result of the block.
// ---------------------------------------------------------------------------------
struct Words4 {
    uint32_t w[4];
};

// Rotate-half (NeoX) pairing, four pairs: A0/B0 hold elements (2m, 2m+1) of the two
// halves for one m, A1/B1 for the next; e0..e3 are the entries of those four pairs
// in order.  Returns the rotated A0, B0, A1, B1 (rounded to bf16, RNE).
__device__ __forceinline__ Words4 rot4_neox(uint32_t A0, uint32_t B0, uint32_t A1, uint32_t B1, uint32_t e0,
                                            uint32_t e1, uint32_t e2, uint32_t e3) {
    uint32_t p0, p1, p2, p3, q0, q1, q2, q3;
    float x0, y0, x1, y1, x2, y2, x3, y3;
    asm("v_perm_b32 %[p0], %[B0], %[A0], %[slo]\n\t"   // (x_2m, y_2m)
        "v_perm_b32 %[q0], %[A0], %[B0], %[slo]\n\t"   // (y_2m, x_2m)
        "v_perm_b32 %[p1], %[B0], %[A0], %[shi]\n\t"
        "v_perm_b32 %[q1], %[A0], %[B0], %[shi]\n\t"
        "v_perm_b32 %[p2], %[B1], %[A1], %[slo]\n\t"
        "v_perm_b32 %[q2], %[A1], %[B1], %[slo]\n\t"
        "v_perm_b32 %[p3], %[B1], %[A1], %[shi]\n\t"
        "v_perm_b32 %[q3], %[A1], %[B1], %[shi]\n\t"
        "v_dot2_f32_bf16 %[x0], %[p0], %[e0], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y0], %[q0], %[e0], 0\n\t"
        "v_dot2_f32_bf16 %[x1], %[p1], %[e1], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y1], %[q1], %[e1], 0\n\t"
        "v_dot2_f32_bf16 %[x2], %[p2], %[e2], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y2], %[q2], %[e2], 0\n\t"
        "v_dot2_f32_bf16 %[x3], %[p3], %[e3], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y3], %[q3], %[e3], 0\n\t"
        "v_cvt_pk_bf16_f32 %[A0], %[x0], %[x1]\n\t"
        "v_cvt_pk_bf16_f32 %[B0], %[y0], %[y1]\n\t"
        "v_cvt_pk_bf16_f32 %[A1], %[x2], %[x3]\n\t"
        "v_cvt_pk_bf16_f32 %[B1], %[y2], %[y3]"
        : [A0] "+v"(A0), [B0] "+v"(B0), [A1] "+v"(A1), [B1] "+v"(B1), [p0] "=&v"(p0), [p1] "=&v"(p1),
          [p2] "=&v"(p2), [p3] "=&v"(p3), [q0] "=&v"(q0), [q1] "=&v"(q1), [q2] "=&v"(q2), [q3] "=&v"(q3),
          [x0] "=&v"(x0), [y0] "=&v"(y0), [x1] "=&v"(x1), [y1] "=&v"(y1), [x2] "=&v"(x2), [y2] "=&v"(y2),
          [x3] "=&v"(x3), [y3] "=&v"(y3)
        : [e0] "v"(e0), [e1] "v"(e1), [e2] "v"(e2), [e3] "v"(e3), [slo] "s"(0x05040100u), [shi] "s"(0x07060302u));
    return Words4{{A0, B0, A1, B1}};
}

// Interleaved (GPT-J) pairing, four pairs: w_i holds the pair (x, y) itself.
__device__ __forceinline__ Words4 rot4_gptj(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, uint32_t e0,
                                            uint32_t e1, uint32_t e2, uint32_t e3) {
    uint32_t q0, q1, q2, q3;
    float x0, y0, x1, y1, x2, y2, x3, y3;
    asm("v_alignbit_b32 %[q0], %[w0], %[w0], 16\n\t"   // (y, x)
        "v_alignbit_b32 %[q1], %[w1], %[w1], 16\n\t"
        "v_alignbit_b32 %[q2], %[w2], %[w2], 16\n\t"
        "v_alignbit_b32 %[q3], %[w3], %[w3], 16\n\t"
        "v_dot2_f32_bf16 %[x0], %[w0], %[e0], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y0], %[q0], %[e0], 0\n\t"
        "v_dot2_f32_bf16 %[x1], %[w1], %[e1], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y1], %[q1], %[e1], 0\n\t"
        "v_dot2_f32_bf16 %[x2], %[w2], %[e2], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y2], %[q2], %[e2], 0\n\t"
        "v_dot2_f32_bf16 %[x3], %[w3], %[e3], 0 neg_hi:[0,1,0]\n\t"
        "v_dot2_f32_bf16 %[y3], %[q3], %[e3], 0\n\t"
        "v_cvt_pk_bf16_f32 %[w0], %[x0], %[y0]\n\t"
        "v_cvt_pk_bf16_f32 %[w1], %[x1], %[y1]\n\t"
        "v_cvt_pk_bf16_f32 %[w2], %[x2], %[y2]\n\t"
        "v_cvt_pk_bf16_f32 %[w3], %[x3], %[y3]"
        : [w0] "+v"(w0), [w1] "+v"(w1), [w2] "+v"(w2), [w3] "+v"(w3), [q0] "=&v"(q0), [q1] "=&v"(q1),
          [q2] "=&v"(q2), [q3] "=&v"(q3), [x0] "=&v"(x0), [y0] "=&v"(y0), [x1] "=&v"(x1), [y1] "=&v"(y1),
          [x2] "=&v"(x2), [y2] "=&v"(y2), [x3] "=&v"(x3), [y3] "=&v"(y3)
        : [e0] "v"(e0), [e1] "v"(e1), [e2] "v"(e2), [e3] "v"(e3));
    return Words4{{w0, w1, w2, w3}};
}

// (a.lo, b.lo) and (a.hi, b.hi) of two bf16 pairs: the rotate-half pairing brings
// element i of one 8-dim run together with element i of the run half a head
// further; one byte permute each (bytes 0-3 of the selector pick from a, 4-7 from b)
__device__ __forceinline__ uint32_t pair_lo(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x05040100u); }
__device__ __forceinline__ uint32_t pair_hi(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x07060302u); }

// c + a.lo + a.hi for a pair of bf16 values (a dot product with (1, 1), one
// accumulate-in-place instruction)
__device__ __forceinline__ float sum2_bf16(uint32_t a, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, 0x3f803f80u), c,
                                           false);
}

// Round two floats to bf16 (round to nearest even) and pack them, lo first.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

// ---------------------------------------------------------------------------------
// RoPE angles.  Pair i turns by p * omega_i.  The angle is kept as a 64-bit binary
// fraction of a revolution, F_i = frac(omega_i / 2pi) scaled by 2^64 (computed on
// the host from theta, or from explicit frequencies), so p * F_i (mod 2^64) is the
// exact phase of any int32 position (negative ones included) up to the rounding of
// F_i; sin/cos then only see a reduced argument in [-0.5, 0.5) revolutions.  A pair
// with F_i = 0 (past a partial rotary width) turns by nothing.
// ---------------------------------------------------------------------------------
__device__ __forceinline__ void rope_cs(int32_t pos, uint64_t step, float& c, float& s) {
    const uint64_t ph = (uint64_t)(int64_t)pos * step;
    const float r = (float)(int32_t)(ph >> 32) * 0x1p-32f;
    sincospif(2.0f * r, &s, &c);
}

__device__ __forceinline__ void rope_cs_f64(int32_t pos, uint64_t step, double& c, double& s) {
    const uint64_t ph = (uint64_t)(int64_t)pos * step;
    const double r = (double)(int64_t)ph * 0x1p-64;
    sincospi(2.0 * r, &s, &c);
}

// Model chunk (8 elements) read into kernel-layout chunk c of q or K.
__device__ __forceinline__ int model_chunk(uint64_t map, int c) { return (int)((map >> (4 * c)) & 15); }

// Table entries: float32 kernels read (cos, sin) as two floats; bf16 kernels read
// (cos, sin) as one bf16 pair, so that rotating a pair (x, y) is two 2-element dot
// products: x' = (x, y).(c, -s) with the sign folded into the instruction, and
// y' = (y, x).(c, s).
__device__ __forceinline__ uint32_t bf16_entry(float c, float s) { return pack_bf16(c, s); }

// cos/sin of N consecutive frequencies i0 .. i0+N-1 (i0 a multiple of 4) at
// position pos from a bf16 table when pos is inside it, else computed.
template <int N, bool TABLE>
__device__ __forceinline__ void rope_cs_n(const float* __restrict__ table, int rope_len, int half,
                                          const uint64_t* fstep, int32_t pos, int i0, float* c, float* s) {
    if (TABLE && (uint32_t)pos < (uint32_t)rope_len) {
        const u32x4_t* t = reinterpret_cast<const u32x4_t*>(reinterpret_cast<const uint32_t*>(table) + (size_t)pos * half + i0);
#pragma unroll
        for (int k = 0; k < N / 4; ++k) {
            const u32x4_t v = t[k];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                c[4 * k + j] = bf_lo(v[j]);
                s[4 * k + j] = bf_hi(v[j]);
            }
        }
    } else {
#pragma unroll
        for (int k = 0; k < N; ++k) rope_cs(pos, fstep[i0 + k], c[k], s[k]);
    }
}

// ---------------------------------------------------------------------------------
// kv_write: one workgroup per new row (its slot read once through the scalar unit),
// one thread per 16-byte chunk of the row's K and V (2^cph_log2 chunks per head).
// ---------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) kv_write_kernel(u32x4_t* __restrict__ k_pool, u32x4_t* __restrict__ v_pool,
                                                       const u32x4_t* __restrict__ k_new,
                                                       const u32x4_t* __restrict__ v_new,
                                                       const int32_t* __restrict__ slots, int cph_log2, int hkv) {
    const int64_t row = blockIdx.x;
    const int per_row = hkv << cph_log2;
    // the thread's first chunk is read together with the slot (one round trip)
    const int c0 = threadIdx.x;
    u32x4_t k0 = u32x4_t{0, 0, 0, 0}, v0 = u32x4_t{0, 0, 0, 0};
    if (c0 < per_row) {
        k0 = k_new[row * per_row + c0];
        v0 = v_new[row * per_row + c0];
    }
    const int32_t slot = __builtin_amdgcn_readfirstlane(slots[row]);
    if (slot < 0) return;
    const int64_t page = ((int64_t)(slot >> 4) * hkv * kBlock + (slot & 15)) << cph_log2;
    auto dst_of = [&](int c) {
        const int h = c >> cph_log2, cc = c & ((1 << cph_log2) - 1);
        return page + ((int64_t)h * kBlock << cph_log2) + cc;
    };
    if (c0 < per_row) {
        k_pool[dst_of(c0)] = k0;
        v_pool[dst_of(c0)] = v0;
    }
    for (int c = c0 + (int)blockDim.x; c < per_row; c += blockDim.x) {
        k_pool[dst_of(c)] = k_new[row * per_row + c];
        v_pool[dst_of(c)] = v_new[row * per_row + c];
    }
}

// ---------------------------------------------------------------------------------
// blocks_copy: one workgroup per cache block, 16-byte chunks of its K and V page
// runs between the pool and a dense [n][page] buffer (gather: pool -> buffer,
// scatter: buffer -> pool).
// ---------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) blocks_copy_kernel(u32x4_t* __restrict__ k_pool, u32x4_t* __restrict__ v_pool,
                                                          u32x4_t* __restrict__ k_buf, u32x4_t* __restrict__ v_buf,
                                                          const int32_t* __restrict__ block_ids, int64_t chunks,
                                                          bool to_pool) {
    const int64_t i = blockIdx.x;
    const int64_t b = block_ids[i];
    u32x4_t* pk = k_pool + b * chunks;
    u32x4_t* pv = v_pool + b * chunks;
    u32x4_t* bk = k_buf + i * chunks;
    u32x4_t* bv = v_buf + i * chunks;
    // four chunks of K and four of V in flight per thread before any store
    const int64_t step = blockDim.x;
    int64_t c = threadIdx.x;
    for (; c + 3 * step < chunks; c += 4 * step) {
        u32x4_t kr[4], vr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            kr[u] = to_pool ? bk[c + u * step] : pk[c + u * step];
            vr[u] = to_pool ? bv[c + u * step] : pv[c + u * step];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (to_pool) {
                pk[c + u * step] = kr[u];
                pv[c + u * step] = vr[u];
            } else {
                bk[c + u * step] = kr[u];
                bv[c + u * step] = vr[u];
            }
        }
    }
    for (; c < chunks; c += step) {
        if (to_pool) {
            pk[c] = bk[c];
            pv[c] = bv[c];
        } else {
            bk[c] = pk[c];
            bv[c] = pv[c];
        }
    }
}

// ---------------------------------------------------------------------------------
// rope_table: entry [p][i] from cos/sin(p * omega_i) in float64, stored as float32
// (cos, sin) or as a bf16 pair (cos, sin).
// ---------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) rope_table_kernel(void* __restrict__ table, int n_pos, int half,
                                                         RopeSteps steps, bool bf16_pairs) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)n_pos * half) return;
    const int p = (int)(idx / half), i = (int)(idx - (int64_t)p * half);
    double c, s;
    rope_cs_f64(p, steps.s[i], c, s);
    if (bf16_pairs)
        static_cast<uint32_t*>(table)[idx] = bf16_entry((float)c, (float)s);
    else
        static_cast<uint2*>(table)[idx] = make_uint2(__float_as_uint((float)c), __float_as_uint((float)s));
}

// ---------------------------------------------------------------------------------
// rope_rotate: x[row][h][:] <- R_{pos[row]} x[row][h][:], one thread per pair.
// ---------------------------------------------------------------------------------
template <typename T, int STYLE>
__global__ void __launch_bounds__(256) rope_rotate_kernel(T* __restrict__ x, int64_t n_pairs, int heads, int d,
                                                          int rot_half, RopeSteps steps,
                                                          const int32_t* __restrict__ positions,
                                                          const void* __restrict__ table, int rope_len) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= n_pairs) return;
    const int half = d / 2;
    const int64_t rh = idx / half;                 // row * heads + h
    const int i = (int)(idx - rh * half);
    if (i >= rot_half) return;                     // past the rotary width: unchanged
    const int32_t pos = positions[rh / heads];
    float c, s;
    if (table != nullptr && (uint32_t)pos < (uint32_t)rope_len) {
        if (sizeof(T) == 4) {
            const uint2 v = static_cast<const uint2*>(table)[(size_t)pos * half + i];
            c = __uint_as_float(v.x);
            s = __uint_as_float(v.y);
        } else {
            const uint32_t v = static_cast<const uint32_t*>(table)[(size_t)pos * half + i];
            c = bf_lo(v);
            s = bf_hi(v);
        }
    } else {
        rope_cs(pos, steps.s[i], c, s);
    }
    T* row = x + rh * d;
    const int ia = STYLE == kNeox ? i : 2 * i, ib = STYLE == kNeox ? i + rot_half : 2 * i + 1;
    const float a = (float)row[ia], b = (float)row[ib];
    row[ia] = (T)(a * c - b * s);
    row[ib] = (T)(b * c + a * s);
}

// A wave-uniform element read through the scalar unit (the value lands in an
// SGPR and waits on the scalar counter, not on the vector-memory queue).
typedef __attribute__((address_space(4))) const int32_t const_i32_t;
__device__ __forceinline__ int32_t scalar_load(const int32_t* p, int i) { return ((const_i32_t*)p)[i]; }

// Group of attention block `bid` (MERGE: of merge block `bid`): binary search over
// the groups in the kernel arguments, or two scalar loads from the table the
// plan-upload launches wrote for a large batch.
template <bool MERGE>
__device__ __forceinline__ Group group_of(const Plan& plan, int bid) {
    if (plan.table != nullptr) {
        const int gi = scalar_load(MERGE ? plan.merge_map : plan.item_map, bid);
        const int32_t* src = reinterpret_cast<const int32_t*>(plan.table + gi);
        Group g;
        int32_t* dst = reinterpret_cast<int32_t*>(&g);
#pragma unroll
        for (int k = 0; k < (int)(sizeof(Group) / 4); ++k) dst[k] = scalar_load(src, k);
        return g;
    }
    return plan.g[MERGE ? plan_search<&Group::merge_base>(plan, bid) : plan_search<&Group::item_base>(plan, bid)];
}

// ---------------------------------------------------------------------------------
// plan_upload: block i writes group first + i of a large batch into the table and
// its index into the block -> group maps of the attention and merge launches.
// ---------------------------------------------------------------------------------
__global__ void __launch_bounds__(256) plan_upload_kernel(const PlanUpload u) {
    const int i = blockIdx.x;
    const Group& g = u.g[i];
    const int item_end = i + 1 < u.n ? u.g[i + 1].item_base : u.item_end;
    const int merge_end = i + 1 < u.n ? u.g[i + 1].merge_base : u.merge_end;
    const int gi = u.first + i;
    if (threadIdx.x < sizeof(Group) / 4)
        reinterpret_cast<int32_t*>(u.table + gi)[threadIdx.x] = reinterpret_cast<const int32_t*>(&g)[threadIdx.x];
    for (int b = g.item_base + (int)threadIdx.x; b < item_end; b += blockDim.x) u.item_map[b] = gi;
    for (int b = g.merge_base + (int)threadIdx.x; b < merge_end; b += blockDim.x) u.merge_map[b] = gi;
}

constexpr int kWaves = kTileRows / 32;   // wave w owns rows [32w, 32w+32); 2 waves per SIMD
constexpr int kThreads = kWaves * 64;

// max over lanes l and l^32 (one VALU permute, no LDS round trip)
__device__ __forceinline__ float max_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

// XOR swizzle of the 16-byte chunks of LDS row `key`.  D = 128: 16 consecutive keys
// get 16 different patterns (conflict-free K operand reads) and 4 consecutive keys
// land in 4 different aligned groups of 4 chunks (conflict-free transposing V reads).
// D = 64 (two rows per bank line): 16 consecutive keys cover both halves x 8 chunks.
template <int D>
__device__ __forceinline__ int swz(int key) {
    if (D == 128) return ((key & 3) << 2) | ((key >> 2) & 3);
    return (key >> 1) & 7;
}

// The decode kernel's 16-key tiles: D = 128 puts key bits 0-1 on chunk bits 2-3,
// key bit 2 on chunk bit 1 and key bit 3 on chunk bit 0.  The 16 keys still get 16
// different patterns (conflict-free K operand reads), and the transposing V reads
// of 8 consecutive keys x 2 chunk halves (a 32-lane pass) cover all 16 chunks once.
template <int D>
__device__ __forceinline__ int dswz(int key) {
    if (D == 128) return ((key & 3) << 2) | (((key >> 2) & 1) << 1) | ((key >> 3) & 1);
    return swz<D>(key);
}

typedef __attribute__((address_space(3))) const uint16_t lds_u16_t;

// an LDS array element as an LDS-space pointer (constant offsets then fold into
// the instruction's offset field)
__device__ __forceinline__ lds_u16_t* as_lds(const uint16_t* p) { return (lds_u16_t*)p; }

// Transposing LDS read: within each 16-lane group, lane i receives element i%4 of
// the 8-byte rows that lanes i/4, i/4+4, i/4+8, i/4+12 point at.
__device__ __forceinline__ s16x4_t lds_read_tr(lds_u16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
}

// One thread's share of a K tile in flight when K is rotated on its way to LDS:
// 16 elements of one key (NeoX: 8 from each half; GPT-J: 16 consecutive) and the
// bf16 (cos, sin) entries of their 8 pairs.
struct TileRegs {
    u32x4_t k[2];
    u32x4_t cs[2];
    int32_t pos;
    int32_t phys;
    bool ok;
};

// wait until this wave's global loads (including loads into LDS) have landed
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// s_waitcnt on vector memory only: wait until at most N loads of this wave are
// outstanding (they complete in issue order)
template <int N>
__device__ __forceinline__ void wait_vmem_n() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((address_space(3))) void lds_void_t;

// Global -> LDS copies written as inline assembly (global_load_lds_dword[x4], LDS
// base in M0): the compiler does not see their LDS writes, so it adds no
// vector-memory waits of its own before later LDS reads -- which it would do for
// every LDS read after the builtin form, draining the whole prefetch queue.  The
// kernel itself waits for them (wait_vmem_n, then a barrier) before reading what
// they wrote.  `lds_wave_base` is wave-uniform; lane i writes bytes
// [size*i, size*(i+1)) after it.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const lds_void_t*)p);
}
__device__ __forceinline__ void dma_lds16(const void* src, const void* lds_wave_base) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(lds_offset(lds_wave_base)) : "memory");
}
__device__ __forceinline__ void dma_lds4(const void* src, const void* lds_wave_base) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(src), "{m0}"(lds_offset(lds_wave_base)) : "memory");
}

// Workgroup barrier that leaves the vector-memory queue alone (__syncthreads
// would also drain every outstanding global->LDS load): this wave's LDS writes are
// waited for, and the compiler may move no memory access across it.
__device__ __forceinline__ void barrier_keep_vmem() {
    __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4));   // lgkmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}


// ---------------------------------------------------------------------------------
// prefill_bf16
//
// Workgroup: 8 waves over up to 256 query rows (token x query head of one KV head's
// group); wave w owns rows [32w, 32w+32) as the 32 columns of its MFMA tiles.
// Per 64-key tile (double-buffered in LDS, the next tile's global loads in flight
// while the current one is consumed):
//   ks[64][D]  rotated K, bf16, 16-byte chunks XOR-swizzled by key;
//   vs[64][D]  V as stored (bf16), same swizzle.
//   S^T (64 keys x 32 queries) = K Q^T: A = K from LDS, B = Q in registers, as two
//   32-key halves whose MFMA chains interleave.  After the MFMA lane l holds query
//   l%32 and keys 8*(j/4) + 4*(l/32) + j%4 (j = 0..15) of each half, so row
//   statistics need one exchange with lane l^32, and one softmax decision covers the
//   tile.  Those probabilities, in that key order, are the B operand of O^T = V^T P^T
//   for 16-key steps; the matching A operand (32 dims x the same 8 keys per lane)
//   comes straight from the untransposed V tile through ds_read_b64_tr_b16.
// ---------------------------------------------------------------------------------
template <int D, int STYLE, bool ROPE, bool TABLE>
__global__ void __launch_bounds__(kThreads, 512 / kThreads) prefill_bf16(const Plan plan, const Args a) {
    constexpr int KD = D / 16;    // 16-wide contraction steps of QK^T
    constexpr int DB = D / 32;    // 32-row blocks of O^T
    constexpr int CH = D / 8;     // 16-byte chunks per row
    constexpr int HALF = D / 2;
    constexpr int BN = kTileKeys;
    constexpr int TPK = D / 16;   // staging threads per key
    constexpr int NSTAGE = BN * TPK;
    constexpr int SU = NSTAGE > kThreads ? NSTAGE / kThreads : 1;   // staged keys per thread
    constexpr int NH = BN / 32;                                      // 32-key halves per tile
    static_assert(BN % 32 == 0 && (NSTAGE <= kThreads || NSTAGE % kThreads == 0), "tile shape");

    __shared__ __attribute__((aligned(16))) uint16_t ks[2][BN * D];
    __shared__ __attribute__((aligned(16))) uint16_t vs[2][BN * D];
    __shared__ uint64_t fstep[HALF];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;

    const int bid = blockIdx.x;
    const Group g = group_of<false>(plan, bid);
    const int part_base = g.part_base;
    const int G = a.group;
    const int n_clusters = a.hkv * g.n_split;
    const int li = bid - g.item_base;
    if (li >= n_clusters * g.n_rt) return;
    int cluster, rt;
    if ((a.hkv & 7) == 0) {
        // blocks bid, bid+8, ... run on one XCD: give them every (split, row tile) of
        // one KV head, so that the row tiles share K/V and the splits share Q in that
        // XCD's L2
        const int per_kvh = g.n_split * g.n_rt;
        const int x = li & 7, k = li >> 3;
        const int kv = x + 8 * (k / per_kvh), r = k % per_kvh;
        cluster = kv * g.n_split + r / g.n_rt;
        rt = r % g.n_rt;
    } else if ((n_clusters & 7) == 0) {
        // the same for the row tiles of one (KV head, split)
        const int x = li & 7, k = li >> 3;
        cluster = x + 8 * (k / g.n_rt);
        rt = k % g.n_rt;
    } else {
        cluster = li / g.n_rt;
        rt = li % g.n_rt;
    }
    const int kvh = cluster / g.n_split, split = cluster - kvh * g.n_split;
    const int rows_total = g.n_tok * G;
    const int row_lo = rt * kTileRows;
    const int row_hi = min(row_lo + kTileRows, rows_total);
    const int t_last = g.tok0 + (row_hi - 1) / G;
    const int kv_lo = g.win + split * g.split_keys;
    const int kv_hi = min(kv_lo + g.split_keys, t_last + 1);
    if (kv_lo >= kv_hi) return;

    // phase steps of the in-kernel cos/sin: staged in LDS when every position needs
    // them (no table); with a table only positions outside it read them, from the
    // kernel arguments
    if (ROPE && !TABLE) {
        for (int i = tid; i < HALF; i += kThreads) fstep[i] = a.fstep[i];
    }
    const uint64_t* fsteps = TABLE ? a.fstep : fstep;

    // ---- queries: rotate at their positions, scale by softmax_scale*log2(e), bf16
    const int wave_row0 = row_lo + wave * 32;
    const bool wave_live = wave_row0 < row_hi;
    const int wave_tmin = g.tok0 + min(wave_row0, row_hi - 1) / G;
    const int row = wave_row0 + l32;
    const bool row_valid = row < row_hi;
    const int toff = row_valid ? row / G : 0;
    const int hl = row_valid ? row - toff * G : 0;
    const int row_tok = row_valid ? g.tok0 + toff : t_last;
    bf16x8_t qb[KD];
    u32x4_t qraw[KD];
    int32_t qpos = 0;
    auto q_issue = [&]() {   // the queries' loads, issued before anything waits
        const uint16_t* qp = static_cast<const uint16_t*>(a.q) +
                             ((size_t)(g.q_row0 + toff) * a.hq + (size_t)kvh * G + hl) * D;
#pragma unroll
        for (int kd = 0; kd < KD; ++kd)   // KD loads on every lane (a row past the tile reads the group's first)
            qraw[kd] = *reinterpret_cast<const u32x4_t*>(qp + model_chunk(a.chunk_map, 2 * kd + hi) * 8);
        if (ROPE && row_valid) qpos = a.positions[g.pos_off + g.tok0 + toff];
    };
    auto q_finish = [&]() {   // rotate, scale by softmax_scale*log2(e), round to bf16
        float xf[KD][8];
#pragma unroll
        for (int kd = 0; kd < KD; ++kd)
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const uint32_t w = row_valid ? qraw[kd][m] : 0u;
                xf[kd][2 * m] = bf_lo(w);
                xf[kd][2 * m + 1] = bf_hi(w);
            }
        if (ROPE) {
            const int32_t pos = qpos;
            if (STYLE == kNeox) {
#pragma unroll
                for (int kd = 0; kd < KD / 2; ++kd) {
                    float c[8], s[8];
                    rope_cs_n<8, TABLE>(a.rope_table, a.rope_len, HALF, fsteps, pos, kd * 16 + 8 * hi, c, s);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float x = xf[kd][e], y = xf[kd + KD / 2][e];
                        xf[kd][e] = x * c[e] - y * s[e];
                        xf[kd + KD / 2][e] = y * c[e] + x * s[e];
                    }
                }
            } else {
#pragma unroll
                for (int kd = 0; kd < KD; ++kd) {
                    float c[4], s[4];
                    rope_cs_n<4, TABLE>(a.rope_table, a.rope_len, HALF, fsteps, pos, kd * 8 + 4 * hi, c, s);
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const float x = xf[kd][2 * m], y = xf[kd][2 * m + 1];
                        xf[kd][2 * m] = x * c[m] - y * s[m];
                        xf[kd][2 * m + 1] = y * c[m] + x * s[m];
                    }
                }
            }
        }
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) {
            u32x4_t w;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                w[m] = pack_bf16(xf[kd][2 * m] * a.scale_log2, xf[kd][2 * m + 1] * a.scale_log2);
            qb[kd] = __builtin_bit_cast(bf16x8_t, w);
        }
    };

    f32x16_t acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = f32x16_t{};
    float m_run = kNegBig, l_run = 0.f;
    // The S^T chain starts from nbias = -m_run (0 while m_run is kNegBig, i.e. no
    // visible key yet), so that it returns the scores relative to the reference
    // maximum and the exponentials need no subtraction; `thr` is the shifted
    // maximum above which the reference moves (8, or any score before the first).
    f32x16_t nbias = f32x16_t{};
    float thr = kNegBig;

    const int32_t* btab = a.block_tables + (size_t)g.req * a.max_blocks;
    const uint16_t* kpool = static_cast<const uint16_t*>(a.k_pool);
    const uint16_t* vpool = static_cast<const uint16_t*>(a.v_pool);

    // staging role of this thread (K through registers when it is rotated): keys
    // kk + u * (kThreads / TPK), u < SU, of every tile, 16-element slice sc
    const bool stager = ROPE && tid < NSTAGE;
    const int kk = tid / TPK, sc = tid - (tid / TPK) * TPK;
    constexpr int KSTEP = kThreads / TPK;
    const int kt0 = kv_lo & ~(kBlock - 1);
    const int n_tiles = (kv_hi - kt0 + BN - 1) / BN;
    // direct global->LDS role (V always, K too without RoPE): lane `lane` of wave
    // `wave` fills 16-byte chunk p = (DPW*wave + i)*64 + lane of the tile, i.e. row
    // p / CH, physical chunk p % CH, which holds logical chunk (p % CH) ^ swz(row)
    constexpr int DPW = BN * CH / (64 * kWaves);
    static_assert(kWaves >= 2, "metadata copies use two waves");
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    auto dkey = [&](int i) { return ((DPW * wave_u + i) * 64 + lane) / CH; };
    auto dchunk = [&](int i) {
        const int p = (DPW * wave_u + i) * 64 + lane;
        return (p % CH) ^ swz<D>(p / CH);
    };

    // per-key metadata two tiles ahead of its use, copied global->LDS with no
    // register round trip (so no load waits on it): the positions of the tile's 64
    // keys (wave 0) and its 4 block ids (wave 1), from keys clamped into the window
    // -- a key outside [kv_lo, kv_hi) stands for the tile's first visible key, so
    // that nothing outside the window is ever read (its score is masked).
    __shared__ int32_t mpos[2][BN];
    __shared__ int32_t mblk[2][BN / kBlock];
    auto clamp_key = [&](int kt, int j) { return (j >= kv_lo && j < kv_hi) ? j : max(kt, kv_lo); };
    auto dma_meta = [&](int t) {
        if (t >= n_tiles) return;
        const int kt = kt0 + t * BN;
        if (ROPE && wave_u == 0) {
            dma_lds4(a.positions + g.pos_off + clamp_key(kt, kt + lane), &mpos[t & 1][0]);
        } else if (wave_u == 1 && lane < BN / kBlock) {
            const int blk = min((kt >> 4) + lane, (kv_hi - 1) >> 4);
            dma_lds4(btab + blk, &mblk[t & 1][0]);
        }
    };
    // every copy's row offset first (the block ids are LDS reads, and no read can pass
    // a copy instruction, so reading them between copies would serialise one LDS
    // round trip per copy), then the copies back to back
    // A tile that lies wholly inside the window needs no clamping: a copy's row is
    // then its block id times the block stride plus a per-lane constant.
    const size_t blk_stride = (size_t)a.hkv * kBlock * D;
    uint32_t lane_off[DPW];
#pragma unroll
    for (int i = 0; i < DPW; ++i) lane_off[i] = (uint32_t)((kvh * kBlock + (dkey(i) & 15)) * D + dchunk(i) * 8);
    auto full_tile = [&](int kt) { return kt >= kv_lo && kt + BN <= kv_hi; };
    auto issue_direct = [&](int t, int buf) {
        const int kt = kt0 + t * BN;
        size_t row_off[DPW];
        if (full_tile(kt)) {
#pragma unroll
            for (int i = 0; i < DPW; ++i)
                row_off[i] = (size_t)(uint32_t)mblk[t & 1][dkey(i) >> 4] * blk_stride + lane_off[i];
        } else {
#pragma unroll
            for (int i = 0; i < DPW; ++i) {
                const int jj = clamp_key(kt, kt + dkey(i));
                const int phys = mblk[t & 1][(jj - kt) >> 4];
                row_off[i] = (((size_t)phys * a.hkv + kvh) * kBlock + (jj & 15)) * D + dchunk(i) * 8;
            }
        }
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
            const int lds_off = (DPW * wave_u + i) * 64 * 8;
            dma_lds16(vpool + row_off[i], &vs[buf][lds_off]);
            if (!ROPE) dma_lds16(kpool + row_off[i], &ks[buf][lds_off]);
        }
    };
    auto load_meta = [&](int t, TileRegs* rr) {
        if (!stager) return;
#pragma unroll
        for (int u = 0; u < SU; ++u) {
            TileRegs& r = rr[u];
            const int kr = kk + u * KSTEP;
            r.pos = mpos[t & 1][kr];
            r.phys = mblk[t & 1][kr >> 4];
        }
    };
    // this thread's two K chunks within its key's row of a block (tiles start on block
    // boundaries and KSTEP is a multiple of the block size, so the row within the
    // block is the same for every tile and every u)
    uint32_t k_off2[2];
    {
        const uint32_t row = (uint32_t)((kvh * kBlock + (kk & 15)) * D);
        k_off2[0] = row + (STYLE == kNeox ? model_chunk(a.chunk_map, sc) * 8 : sc * 16);
        k_off2[1] = row + (STYLE == kNeox ? model_chunk(a.chunk_map, sc + CH / 2) * 8 : sc * 16 + 8);
    }
    auto load_tile = [&](int t, TileRegs* rr) {
        if (!stager) return;
#pragma unroll
        for (int u = 0; u < SU; ++u) {
        TileRegs& r = rr[u];
        const int kr = kk + u * KSTEP;
        const int j = kt0 + t * BN + kr;
        r.ok = j >= kv_lo && j < kv_hi;
        r.k[0] = r.k[1] = u32x4_t{0, 0, 0, 0};
        if (r.ok) {
            const uint16_t* kp = kpool + (size_t)(uint32_t)r.phys * blk_stride;
            r.k[0] = *reinterpret_cast<const u32x4_t*>(kp + k_off2[0]);
            r.k[1] = *reinterpret_cast<const u32x4_t*>(kp + k_off2[1]);
            if (TABLE && (uint32_t)r.pos < (uint32_t)a.rope_len) {
                const u32x4_t* tp = reinterpret_cast<const u32x4_t*>(reinterpret_cast<const uint32_t*>(a.rope_table) +
                                                                     (size_t)r.pos * HALF + sc * 8);
                r.cs[0] = tp[0];
                r.cs[1] = tp[1];
            }
        }
        }
    };
    auto store_tile = [&](int buf, TileRegs* rr) {
        if (!stager) return;
#pragma unroll
        for (int u = 0; u < SU; ++u) {
        TileRegs& r = rr[u];
        const int kr = kk + u * KSTEP;
        // e[k] = (cos, sin) of pair sc*8 + k as bf16: from the table, or computed for
        // keys whose position lies outside it (a wave-uniform branch, so the common
        // all-in-table case runs no fallback code)
        uint32_t e[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) e[k] = r.cs[k / 4][k % 4];
        const bool need_cs = r.ok && !(TABLE && (uint32_t)r.pos < (uint32_t)a.rope_len);
        if (!TABLE || __builtin_amdgcn_ballot_w64(need_cs) != 0) {
            if (need_cs) {
                if (TABLE) {
                    // rare: one compact loop, each new entry shifted in at the end of the
                    // window, keeps the code inside the tile loop small
#pragma unroll 1
                    for (int k = 0; k < 8; ++k) {
                        float c, sn;
                        rope_cs(r.pos, fsteps[sc * 8 + k], c, sn);
#pragma unroll
                        for (int m = 0; m < 7; ++m) e[m] = e[m + 1];
                        e[7] = bf16_entry(c, sn);
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        float c, sn;
                        rope_cs(r.pos, fsteps[sc * 8 + k], c, sn);
                        e[k] = bf16_entry(c, sn);
                    }
                }
            }
        }
        if (STYLE == kNeox) {
            // r.k[0][m] = (x_2m, x_2m+1), r.k[1][m] = (y_2m, y_2m+1)
#pragma unroll
            for (int m = 0; m < 4; m += 2) {
                const Words4 o = rot4_neox(r.k[0][m], r.k[1][m], r.k[0][m + 1], r.k[1][m + 1], e[2 * m], e[2 * m + 1],
                                           e[2 * m + 2], e[2 * m + 3]);
                r.k[0][m] = o.w[0];
                r.k[1][m] = o.w[1];
                r.k[0][m + 1] = o.w[2];
                r.k[1][m + 1] = o.w[3];
            }
        } else {
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const Words4 o = rot4_gptj(r.k[h2][0], r.k[h2][1], r.k[h2][2], r.k[h2][3], e[4 * h2], e[4 * h2 + 1],
                                           e[4 * h2 + 2], e[4 * h2 + 3]);
#pragma unroll
                for (int m = 0; m < 4; ++m) r.k[h2][m] = o.w[m];
            }
        }
        // a key outside the window (partial tiles only) was loaded as zeros and its
        // entries e are finite (the table's, or the last tile's, or zero), so it is
        // stored as zeros; its score is masked in any case
        const int sw = swz<D>(kr);
        uint16_t* krow = &ks[buf][kr * D];
        const int ca = STYLE == kNeox ? sc : 2 * sc;
        const int cb = STYLE == kNeox ? sc + CH / 2 : 2 * sc + 1;
        *reinterpret_cast<u32x4_t*>(krow + ((ca ^ sw) << 3)) = r.k[0];
        *reinterpret_cast<u32x4_t*>(krow + ((cb ^ sw) << 3)) = r.k[1];
        }
    };

    // ---- prologue: the queries' loads and the first tile's loads are all in flight
    // before the first wait
    TileRegs regs[SU];
#pragma unroll
    for (int u = 0; u < SU; ++u) regs[u] = TileRegs{};   // entries start finite
    dma_meta(0);
    dma_meta(1);
    q_issue();
    // the metadata copies (issued before the KD query loads, which may still be in
    // flight) have landed, and the phase steps are staged
    wait_vmem_n<KD>();
    barrier_keep_vmem();
    issue_direct(0, 0);
    load_meta(0, regs);
    load_tile(0, regs);
    q_finish();
    store_tile(0, regs);
    wait_vmem();
    __syncthreads();

    // per-lane LDS element offsets, constant over tiles: the K operand row of each
    // contraction step, and the V^T operand rows (keys 4*(l/32)+{0..3} and the same
    // +8 of a 16-key step) of each 32-dim block.  Buffer, 32-key half and 16-key step
    // add compile-time constants (the swizzle only depends on a key's low 4 bits).
    int k_off[KD];
#pragma unroll
    for (int kd = 0; kd < KD; ++kd) k_off[kd] = l32 * D + (((kd * 2 + hi) ^ swz<D>(l32)) << 3);
    int v_off[DB];
    {
        const int q16 = (lane >> 4) & 1, kq = (lane & 15) >> 2, dq = 4 * (lane & 3);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const int key = 4 * hi + kq;
            const int d = db * 32 + q16 * 16 + dq;
            v_off[db] = key * D + (((d >> 3) ^ swz<D>(key)) << 3) + (d & 7);
        }
    }
    // the same lane's row 8 keys further: swz(key + 8) = swz(key) ^ kSwz8
    constexpr int kSwz8 = D == 128 ? 2 : 4;
    static_assert(D == 64 || D == 128, "head_dim");
    const int hi_key = min(kv_hi - 1, row_tok);   // last key this lane's row may see

    auto step = [&](auto bufc, int t) {
        constexpr int buf = decltype(bufc)::value;
        const int kt = kt0 + t * BN;
        const bool more = t + 1 < n_tiles;
        // direct loads of the next tile (no registers) go out first; the rotated-K
        // register loads wait until the score tile is dead (after the softmax)
        if (more) load_meta(t + 1, regs);
        
        dma_meta(t + 2);   // into the slot tile t's metadata has left
        if (more) issue_direct(t + 1, buf ^ 1);
        if (wave_live) {
            const uint16_t* kb = &ks[buf][0];
            lds_u16_t* vb = as_lds(&vs[buf][0]);
            const bool masked = kt < kv_lo || kt + BN > kv_hi || kt + BN - 1 > wave_tmin;
            // ---- S^T (32 keys x 32 queries) = K Q^T for both halves of the tile, the two
            // MFMA chains interleaved (each accumulator was last written two MFMAs back)
            f32x16_t s[NH];
#pragma unroll
            for (int kd = 0; kd < KD; ++kd)
#pragma unroll
                for (int mb = 0; mb < NH; ++mb) {
                    const bf16x8_t af = *reinterpret_cast<const bf16x8_t*>(kb + k_off[kd] + mb * 32 * D);
                    s[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, qb[kd], kd == 0 ? nbias : s[mb], 0, 0, 0);
                }
            // keep the K operand reads six reads ahead of their MFMAs (left alone, the
            // compiler waits on each read right after issuing it)
#pragma unroll
            for (int i = 0; i < 6; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read
#pragma unroll
            for (int i = 0; i < KD * NH - 6; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                          // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
#pragma unroll
            for (int i = 0; i < 6; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            // ---- window mask on tiles that cross a boundary of the visible set: a bit
            // mask of the visible keys relative to this lane's first key of each half
            if (masked) {
#pragma unroll
                for (int mb = 0; mb < NH; ++mb) {
                    const int base = kt + mb * 32 + 4 * hi;
                    const int lo = max(kv_lo - base, 0), top = min(hi_key - base, 31);
                    const uint32_t upto = (2u << (uint32_t)max(top, 0)) - 1u;
                    const uint32_t vis = (top < lo) ? 0u : (upto & ~((1u << (uint32_t)min(lo, 31)) - 1u));
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int c = 8 * (j >> 2) + (j & 3);
                        s[mb][j] = (vis & (1u << c)) ? s[mb][j] : -INFINITY;
                    }
                }
            }
            // ---- online softmax in the log2 domain, one decision per tile.  The
            // reference maximum only moves when some row's maximum grows by more than 8
            // (probabilities stay below 2^8), so most tiles skip rescaling.
            float mx = kNegBig;
#pragma unroll
            for (int mb = 0; mb < NH; ++mb)
#pragma unroll
                for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[mb][j]);
            mx = max_xor32(mx);
            if (__builtin_amdgcn_ballot_w64(mx > thr) != 0) {
                const float m_off = m_run > kNegBig ? m_run : 0.f;   // what the chain subtracted
                const float m_new = fmaxf(m_run, mx + m_off);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
                l_run *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db) acc[db] *= alpha;
                m_run = m_new;
                const bool seen = m_new > kNegBig;
                const float d = seen ? m_new - m_off : 0.f;
#pragma unroll
                for (int mb = 0; mb < NH; ++mb) s[mb] -= d;
                const float nb = seen ? -m_new : 0.f;
#pragma unroll
                for (int j = 0; j < 16; ++j) nbias[j] = nb;
                thr = seen ? 8.f : kNegBig;
            }
            // probabilities rounded to bf16 for P V; the row sum adds exactly those, two
            // at a time
            bf16x8_t pb[2 * NH];
            float part[2] = {0.f, 0.f};
#pragma unroll
            for (int mb = 0; mb < NH; ++mb)
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    u32x4_t w;
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const float p0 = __builtin_amdgcn_exp2f(s[mb][8 * k2 + 2 * m]);
                        const float p1 = __builtin_amdgcn_exp2f(s[mb][8 * k2 + 2 * m + 1]);
                        w[m] = pack_bf16(p0, p1);
                        part[m & 1] = sum2_bf16(w[m], part[m & 1]);
                    }
                    pb[2 * mb + k2] = __builtin_bit_cast(bf16x8_t, w);
                }
            l_run += part[0] + part[1];
            if (more) load_tile(t + 1, regs);
            // ---- O^T += V^T P^T, 16 keys per step, the DB independent accumulators in turn
#pragma unroll
            for (int k4 = 0; k4 < 2 * NH; ++k4)
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const int row0 = 16 * k4 * D;
                    const s16x4_t both[2] = {lds_read_tr(vb + v_off[db] + row0),
                                             lds_read_tr(vb + (v_off[db] ^ (kSwz8 << 3)) + 8 * D + row0)};
                    acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, both), pb[k4],
                                                                      acc[db], 0, 0, 0);
                }
        }
        if (more) {
            if (!wave_live) load_tile(t + 1, regs);
            store_tile(buf ^ 1, regs);
        }
        wait_vmem();
        __syncthreads();
    };
    for (int t = 0; t < n_tiles; t += 2) {
        step(std::integral_constant<int, 0>{}, t);
        if (t + 1 < n_tiles) step(std::integral_constant<int, 1>{}, t + 1);
    }

    // ---- epilogue: normalise (a split by its own sum, its running maximum and sum
    // stored beside it), round to bf16 and store.  The rows pass through this wave's
    // own 32 rows of the now idle K/V tile buffers (chunks XOR-swizzled by row), so
    // that each global store writes whole 16-byte chunks of 64 / CH complete rows.
    const float lt = sum_xor32(l_run);
    if (!wave_live) return;
    const bool is_split = g.n_split > 1;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    uint16_t* stage = (wave < kWaves / 2 ? &ks[0][0] : &vs[0][0]) + (wave % (kWaves / 2)) * 32 * D;
    static_assert(2 * BN >= 32 * (kWaves / 2), "epilogue staging rows");
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const int c = db * 4 + q4;   // dims 8c .. 8c+7 of the row; this lane holds half of them
            const u32x2_t w = {pack_bf16(acc[db][4 * q4] * inv, acc[db][4 * q4 + 1] * inv),
                               pack_bf16(acc[db][4 * q4 + 2] * inv, acc[db][4 * q4 + 3] * inv)};
            *reinterpret_cast<u32x2_t*>(stage + l32 * D + ((c ^ (l32 & (CH - 1))) << 3) + 4 * hi) = w;
        }
    __builtin_amdgcn_wave_barrier();
    const size_t slot = (size_t)part_base + (size_t)cluster * g.n_rt + rt;
    constexpr int RPI = 64 / CH;   // rows per store instruction
#pragma unroll
    for (int i = 0; i < 32 / RPI; ++i) {
        const int r = i * RPI + lane / CH, c = lane % CH;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(stage + r * D + ((c ^ (r & (CH - 1))) << 3));
        const int rr = wave_row0 + r;
        if (rr >= row_hi) continue;
        uint16_t* dst;
        if (is_split) {
            dst = reinterpret_cast<uint16_t*>(a.part_o) + (slot * kTileRows + (rr - row_lo)) * D;
        } else {
            const int to = rr / G, h = rr - to * G;
            dst = static_cast<uint16_t*>(a.o) + ((size_t)(g.q_row0 + to) * a.hq + (size_t)kvh * G + h) * D;
        }
        *reinterpret_cast<u32x4_t*>(dst + c * 8) = v;
    }
    if (is_split && hi == 0 && row_valid)   // the lane's row is row_lo + 32 wave + l32
        *reinterpret_cast<float2*>(a.part_ml + (slot * kTileRows + (32 * wave_u + (int)(threadIdx.x & 31))) * 2) =
            make_float2(m_run, lt);
}

// ---------------------------------------------------------------------------------
// merge: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s over the non-empty splits
// of one (row tile, KV head), as a streaming log-sum-exp merge.  One block per
// kMergeRows rows, 8 dims (16 bytes of bf16) of a row per thread; the loads of 8 splits are issued
// together before they are combined.
// ---------------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kMergeRows * D / 8) merge_kernel(const Plan plan, const Args a) {
    constexpr int TPR = D / 8;                      // threads per row, 8 dims (16 bytes) each
    constexpr int CHUNKS = kTileRows / kMergeRows;  // blocks per (row tile, KV head)
    constexpr int U = 8;                            // splits loaded per batch
    const Group g = group_of<true>(plan, blockIdx.x);
    const int part_base = g.part_base, merge_base = g.merge_base;
    if (g.n_split <= 1) return;
    int li = blockIdx.x - merge_base;
    if (li >= a.hkv * g.n_rt * CHUNKS) return;
    const int chunk = li % CHUNKS;
    li /= CHUNKS;
    const int kvh = li / g.n_rt, rt = li - (li / g.n_rt) * g.n_rt;
    const int G = a.group;
    const int row_lo = rt * kTileRows;
    const int row_hi = min(row_lo + kTileRows, g.n_tok * G);
    const int t_last = g.tok0 + (row_hi - 1) / G;
    int n_live = 0;
    for (int s = 0; s < g.n_split; ++s)
        if (g.win + s * g.split_keys < t_last + 1) n_live = s + 1;
    const int r = chunk * kMergeRows + (int)threadIdx.x / TPR;
    const int q8 = (int)threadIdx.x % TPR;
    if (row_lo + r >= row_hi) return;
    const size_t slot0 = (size_t)part_base + (size_t)kvh * g.n_split * g.n_rt + rt;
    float M = kNegBig, den = 0.f;
    float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t* part = reinterpret_cast<const uint16_t*>(a.part_o);
    for (int s0 = 0; s0 < n_live; s0 += U) {
        float2 ml[U];
        u32x4_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ml[u] = make_float2(kNegBig, 0.f);
            v[u] = u32x4_t{0, 0, 0, 0};
            if (s0 + u < n_live) {
                const size_t slot = slot0 + (size_t)(s0 + u) * g.n_rt;
                ml[u] = *reinterpret_cast<const float2*>(a.part_ml + (slot * kTileRows + r) * 2);
                v[u] = *reinterpret_cast<const u32x4_t*>(part + (slot * kTileRows + r) * D + q8 * 8);
            }
        }
        // each split's output is normalised: weight it by its sum times 2^(m_s - M)
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (!(ml[u].y > 0.f)) continue;   // split saw no key of this row
            const float m_new = fmaxf(M, ml[u].x);
            const float c_old = __builtin_amdgcn_exp2f(M - m_new);
            const float w = __builtin_amdgcn_exp2f(ml[u].x - m_new) * ml[u].y;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                num[2 * e] = num[2 * e] * c_old + w * bf_lo(v[u][e]);
                num[2 * e + 1] = num[2 * e + 1] * c_old + w * bf_hi(v[u][e]);
            }
            den = den * c_old + w;
            M = m_new;
        }
    }
    const float inv = 1.f / den;
    const int row = row_lo + r;
    const int toff = row / G, hl = row - toff * G;
    u32x4_t out;
#pragma unroll
    for (int e = 0; e < 4; ++e) out[e] = pack_bf16(num[2 * e] * inv, num[2 * e + 1] * inv);
    *reinterpret_cast<u32x4_t*>(static_cast<uint16_t*>(a.o) + ((size_t)(g.q_row0 + toff) * a.hq + (size_t)kvh * G + hl) * D +
                                q8 * 8) = out;
}

// ---------------------------------------------------------------------------------
// one-query (decode) attention: helpers
// ---------------------------------------------------------------------------------
constexpr int kDecKeys = kDecTileKeys;

__device__ __forceinline__ float max_xor16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D, int HW>
constexpr int dec_stages() {
    // K + V of the workgroup's HW heads x 16 keys, plus the tile's cos/sin rows, per
    // stage, within the workgroup's share of 144 KB of LDS
    constexpr int budget = 147456 / dec_wgs_per_cu(HW);
    constexpr int stage = 2 * HW * kDecKeys * D * 2 + kDecKeys * D / 2 * 4;
    return budget / stage > 4 ? 4 : budget / stage;
}

// One pipeline stage of the decode kernel in LDS.  Each stage is its own LDS
// object (as is each stage's position slot) so that reading one stage does not
// make the compiler wait for the global->LDS loads still filling another.
template <int D, bool ROPE, int HW>
struct DecStage {
    uint16_t k[HW * kDecKeys * D];   // [head][key][D], chunks swizzled by key
    uint16_t v[HW * kDecKeys * D];
    uint32_t tab[ROPE ? kDecKeys * D / 2 : 4];  // [key][pair] bf16 (c, s), 16-byte chunks swizzled by key
};

template <int I>
struct Idx {
    static constexpr int value = I;
};

// ---------------------------------------------------------------------------------
// decode_bf16
//
// One query per (request, query head).  Workgroup = HW waves (8, or 2 / 4 when
// the model's KV heads need no more, dec_waves; narrower workgroups take a
// matching share of the CU's LDS, so that several run side by side) = (request,
// key split, group of HH = HW / CB KV heads): a KV head's G <= 64 query heads are
// split over CB = ceil(G / 16) waves (1, 2 or 4), each holding 16 of them as the
// columns of its 16x16 MFMA tiles; wave w owns KV head HH*hg + w / CB and query
// heads 16 (w % CB) ..+15 of its group.  A tile is 16 keys = one cache block, so its K or V
// for the group's heads is one contiguous run of the pool.  Every global read of
// the key loop goes straight to LDS (K unrotated, V, the cos/sin rows of the
// tile's 16 keys, the positions of a later tile), NST tiles deep, so the only wait
// per tile is for the oldest stage.  Each wave rotates its own K operand in
// registers right before the MFMA: with CB = 1 every K element is consumed by
// exactly one wave (the CB waves of a wider query group each rotate it).
//   S^T (16 keys x 16 queries) = K Q^T    v_mfma_f32_16x16x32_bf16
//   O^T (16 dims x 16 queries) += V^T P^T v_mfma_f32_16x16x16_bf16, V^T through
//                                          ds_read_b64_tr_b16
// After QK^T lane l holds query l%16 and keys 4*(l/16) + {0..3}, which is exactly
// the B operand of the PV step, so probabilities never leave their lanes; row
// statistics need two exchanges (lanes l^16 and l^32).
// ---------------------------------------------------------------------------------
template <int D, int STYLE, bool ROPE, bool TABLE, int HW>
__global__ void __launch_bounds__(HW * 64, 1) decode_bf16(const Plan plan, const Args a) {
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    constexpr int KD = D / 32;             // 16x16x32 contraction steps of QK^T
    constexpr int DB = D / 16;             // 16-dim blocks of O^T
    constexpr int CH = D / 8;              // 16-byte chunks per K/V row
    constexpr int HALF = D / 2;
    constexpr int TK = kDecKeys;
    constexpr int NT = HW * 64;            // threads
    constexpr int HSZ = TK * D;            // elements of one head's tile
    constexpr int DPL = HW * HSZ / 8 / NT; // 16-byte direct loads per lane per tile, each of K and V
    constexpr int TROW = HALF / 4;         // 16-byte chunks (4 entries) per cos/sin row
    constexpr int TCH = TK * TROW;         // chunks of the tile's cos/sin rows
    constexpr int NST = dec_stages<D, HW>();   // pipeline stages (tiles resident in LDS)
    constexpr int LPS = 2 * DPL;           // unconditional loads per lane per stage
    static_assert(DPL >= 1 && TROW >= 8 && NST >= 2 && NST <= 4, "decode tile shape");
    static_assert((NST - 2) * LPS < 64, "vmcnt range");
    typedef DecStage<D, ROPE, HW> Stage;

    __shared__ __attribute__((aligned(16))) Stage st0, st1, st2, st3;
    __shared__ int32_t pos0[TK], pos1[TK], pos2[TK], pos3[TK];
    __shared__ uint64_t fstep[HALF];
    auto stage = [&](auto b) -> Stage& {
        constexpr int B = decltype(b)::value % NST;
        if constexpr (B == 0) return st0;
        else if constexpr (B == 1) return st1;
        else if constexpr (B == 2) return st2;
        else return st3;
    };
    auto pslot = [&](auto b) -> int32_t* {
        constexpr int B = decltype(b)::value % NST;
        if constexpr (B == 0) return pos0;
        else if constexpr (B == 1) return pos1;
        else if constexpr (B == 2) return pos2;
        else return pos3;
    };

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c16 = lane & 15, q4 = lane >> 4;   // MFMA column (query / key row) and row group
    const int G = a.group;
    const int CB = dec_col_blocks(G), HH = HW / CB;   // waves per KV head, KV heads per workgroup
    const int kv_slot = wave / CB, qc = (wave % CB) * 16 + c16;   // KV head slot, this lane's query column
    const int n_hg = (a.hkv + HH - 1) / HH;
    const Group g = group_of<false>(plan, blockIdx.x);
    const int part_base = g.part_base;
    const int li = blockIdx.x - g.item_base;
    if (li >= g.n_split * n_hg) return;
    const int split = li / n_hg, hg = li - (li / n_hg) * n_hg;
    const int L = g.tok0 + 1;                    // keys of the request (the query is its last token)
    const int kv_lo = g.win + split * g.split_keys;
    const int kv_hi = min(kv_lo + g.split_keys, L);
    if (kv_lo >= kv_hi) return;
    const int kvh = hg * HH + kv_slot;           // this wave's KV head
    const bool head_live = kvh < a.hkv && qc - c16 < G;   // the head exists and some column is a query
    const int n_heads_here = min(HH, a.hkv - hg * HH);

    if (ROPE)
        for (int i = tid; i < HALF; i += NT) fstep[i] = a.fstep[i];

    const int32_t* btab = a.block_tables + (size_t)g.req * a.max_blocks;
    const uint16_t* kpool = static_cast<const uint16_t*>(a.k_pool);
    const uint16_t* vpool = static_cast<const uint16_t*>(a.v_pool);
    const int kt0 = kv_lo & ~(TK - 1);
    const int n_tiles = (kv_hi - kt0 + TK - 1) / TK;

    // keys outside [kv_lo, kv_hi) are loaded from the tile's first visible key, so
    // that nothing outside the window is read (their scores are masked)
    auto clamp_key = [&](int kt, int j) { return (j >= kv_lo && j < kv_hi) ? j : max(kt, kv_lo); };

    // positions of tile u's 16 keys into position slot B (16 lanes of wave 0)
    auto load_positions = [&](auto b, int u) {
        if (!ROPE || wave != 0 || u >= n_tiles) return;
        if (lane < TK) {
            const int kt = kt0 + u * TK;
            dma_lds4(a.positions + g.pos_off + clamp_key(kt, kt + lane), pslot(b));
        }
    };
    load_positions(Idx<0>{}, 0);
    if constexpr (NST > 2) load_positions(Idx<1>{}, 1);
    if constexpr (NST > 3) load_positions(Idx<2>{}, 2);

    // ---- queries: B operand of S^T = K Q^T, rotated at the last token's position
    bf16x8_t qb[KD];
    {
        const bool qv = head_live && qc < G;
        const int qh = kvh * G + qc;
        const uint16_t* qp = static_cast<const uint16_t*>(a.q) + ((size_t)g.q_row0 * a.hq + qh) * D;
        float xf[KD][8];
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) {
            const u32x4_t raw =
                qv ? *reinterpret_cast<const u32x4_t*>(qp + model_chunk(a.chunk_map, kd * 4 + q4) * 8) : u32x4_t{0, 0, 0, 0};
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                xf[kd][2 * m] = bf_lo(raw[m]);
                xf[kd][2 * m + 1] = bf_hi(raw[m]);
            }
        }
        if (ROPE) {
            const int32_t pos = a.positions[g.pos_off + g.tok0];
            const uint64_t* fs = TABLE ? a.fstep : fstep;
            if (!TABLE) __syncthreads();   // phase steps in LDS
            if (STYLE == kNeox) {
#pragma unroll
                for (int kd = 0; kd < KD / 2; ++kd) {
                    float c[8], sn[8];
                    rope_cs_n<8, TABLE>(a.rope_table, a.rope_len, HALF, fs, pos, kd * 32 + 8 * q4, c, sn);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float x = xf[kd][e], y = xf[kd + KD / 2][e];
                        xf[kd][e] = x * c[e] - y * sn[e];
                        xf[kd + KD / 2][e] = y * c[e] + x * sn[e];
                    }
                }
            } else {
#pragma unroll
                for (int kd = 0; kd < KD; ++kd) {
                    float c[4], sn[4];
                    rope_cs_n<4, TABLE>(a.rope_table, a.rope_len, HALF, fs, pos, kd * 16 + 4 * q4, c, sn);
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const float x = xf[kd][2 * m], y = xf[kd][2 * m + 1];
                        xf[kd][2 * m] = x * c[m] - y * sn[m];
                        xf[kd][2 * m + 1] = y * c[m] + x * sn[m];
                    }
                }
            }
        }
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) {
            u32x4_t w;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                w[m] = pack_bf16(xf[kd][2 * m] * a.scale_log2, xf[kd][2 * m + 1] * a.scale_log2);
            qb[kd] = __builtin_bit_cast(bf16x8_t, w);
        }
    }
    wait_vmem();       // the first positions have landed
    __syncthreads();   // ... for every wave; phase steps staged

    // ---- tile u into stage B = u % NST, all straight into LDS.  Lane `lane` of
    // wave `wave` fills 16-byte chunk p = (i*HW + wave)*64 + lane of the stage's K
    // and V: head p / (HSZ/8), key row, physical chunk pc holding logical chunk
    // pc ^ swz(key).  Chunk c < TCH of the tile's cos/sin rows (key c / TROW,
    // physical chunk pc holding logical chunk pc ^ (key % TROW): conflict-free reads
    // across the keys) comes from the table, or is computed for positions outside it.  The
    // positions of tile u + NST - 1 (the next tile issued after this one) go out
    // first, into the slot tile u - 1 has finished with.
    auto issue_tile = [&](auto b, int u) {
        constexpr int B = decltype(b)::value % NST;
        Stage& sg = stage(b);
        const int kt = kt0 + u * TK;
        load_positions(Idx<B + NST - 1>{}, u + NST - 1);
        if (ROPE) {
            const int32_t* pp = pslot(b);
#pragma unroll
            for (int k = 0; k * NT < TCH; ++k) {
                const int c = k * NT + tid;
                if (c < TCH) {
                    const int tkey = c / TROW, lc = (c % TROW) ^ (tkey & (TROW - 1));
                    const int32_t pos = pp[tkey];
                    const bool in_table = TABLE && (uint32_t)pos < (uint32_t)a.rope_len;
                    if (in_table)
                        dma_lds16(reinterpret_cast<const uint32_t*>(a.rope_table) + (size_t)pos * HALF + 4 * lc,
                                  &sg.tab[(k * NT + wave * 64) * 4]);
                    if (!TABLE || __builtin_amdgcn_ballot_w64(!in_table) != 0) {
                        if (!in_table) {
                            uint32_t w[4] = {0u, 0u, 0u, 0u};
                            if (TABLE) {
                                // rare with a table: a compact loop, entries shifted in
#pragma unroll 1
                                for (int e = 0; e < 4; ++e) {
                                    float ce, se;
                                    rope_cs(pos, fstep[4 * lc + e], ce, se);
                                    w[0] = w[1];
                                    w[1] = w[2];
                                    w[2] = w[3];
                                    w[3] = bf16_entry(ce, se);
                                }
                            } else {
#pragma unroll
                                for (int e = 0; e < 4; ++e) {
                                    float ce, se;
                                    rope_cs(pos, fstep[4 * lc + e], ce, se);
                                    w[e] = bf16_entry(ce, se);
                                }
                            }
                            *reinterpret_cast<u32x4_t*>(&sg.tab[c * 4]) = u32x4_t{w[0], w[1], w[2], w[3]};
                        }
                    }
                }
            }
        }
        const int blk = scalar_load(btab, kt >> 4);   // the tile is exactly one block
#pragma unroll
        for (int i = 0; i < DPL; ++i) {
            const int p = (i * HW + wave) * 64 + lane;
            const int hh = p / (HSZ / 8), q = p % (HSZ / 8);
            const int kk = q / CH, pc = q % CH;
            const int j = clamp_key(kt, kt + kk);
            const int hs = min(hh, n_heads_here - 1);   // heads past Hkv load a real head, never read
            const size_t off = (((size_t)blk * a.hkv + hg * HH + hs) * kBlock + (j & 15)) * D + ((pc ^ dswz<D>(kk)) << 3);
            dma_lds16(kpool + off, &sg.k[(i * HW + wave) * 64 * 8]);
            dma_lds16(vpool + off, &sg.v[(i * HW + wave) * 64 * 8]);
        }
    };

    f32x4_t acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float m_run = kNegBig, l_run = 0.f;

    // per-lane LDS offsets within one head's tile: K operand rows (key c16, logical
    // chunk 4*kd + q4), the cos/sin chunks of the pairs those dims belong to (NeoX:
    // pairs 32*kd + 8*q4 + e, kd < KD/2, 2 chunks each; GPT-J: pairs 16*kd + 4*q4 + e,
    // 1 chunk each), and the transposing V reads (key 4*q4 + (lane%16)/4, dims
    // 16*db + 4*(lane%4))
    int k_off[KD];
#pragma unroll
    for (int kd = 0; kd < KD; ++kd)
        k_off[kd] = kv_slot * HSZ + c16 * D + ((model_chunk(a.chunk_map, kd * 4 + q4) ^ dswz<D>(c16)) << 3);
    constexpr int NTC = KD;   // NeoX: 2 chunks for each of the KD/2 steps; GPT-J: 1 for each of KD
    int t_off[NTC];
#pragma unroll
    for (int u = 0; u < NTC; ++u) {
        const int lc = STYLE == kNeox ? (u / 2) * 8 + 2 * q4 + (u % 2) : u * 4 + q4;
        t_off[u] = c16 * HALF + 4 * (lc ^ (c16 & (TROW - 1)));
    }
    int v_off[DB];
    {
        const int key = 4 * q4 + ((lane & 15) >> 2);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const int d = db * 16 + 4 * (lane & 3);
            v_off[db] = kv_slot * HSZ + key * D + (((d >> 3) ^ dswz<D>(key)) << 3) + (d & 7);
        }
    }

    // ---- one tile of the key loop, stage B = t % NST
    auto step = [&](auto b, int t) {
        Stage& sg = stage(b);
        const int kt = kt0 + t * TK;
        // tile t has landed once no more than the later issued stages' loads are
        // outstanding; the barrier then also frees the stage read at t - 1
        if (t + NST - 2 < n_tiles) wait_vmem_n<(NST - 2) * LPS>();
        else wait_vmem();
        barrier_keep_vmem();
        if (t + NST - 1 < n_tiles) issue_tile(Idx<decltype(b)::value + NST - 1>{}, t + NST - 1);
        if (!head_live) return;
        lds_u16_t* vb = as_lds(sg.v);
        u32x4_t kf[KD];
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) kf[kd] = *reinterpret_cast<const u32x4_t*>(sg.k + k_off[kd]);
        if (ROPE) {
            // rotate the K operand in registers with bf16 entries (c, s)
            u32x4_t te[NTC];
#pragma unroll
            for (int u = 0; u < NTC; ++u) te[u] = *reinterpret_cast<const u32x4_t*>(&sg.tab[t_off[u]]);
            if (STYLE == kNeox) {
                // te[2 kd] and te[2 kd + 1] hold the entries of pairs 0-3 and 4-7 of this
                // lane's 8-pair run; kf[kd][m] = (x_2m, x_2m+1), kf[kd + KD/2][m] = (y_2m, y_2m+1)
#pragma unroll
                for (int kd = 0; kd < KD / 2; ++kd)
#pragma unroll
                    for (int m = 0; m < 4; m += 2) {
                        const u32x4_t ee = te[2 * kd + m / 2];
                        const Words4 o = rot4_neox(kf[kd][m], kf[kd + KD / 2][m], kf[kd][m + 1], kf[kd + KD / 2][m + 1],
                                                   ee[0], ee[1], ee[2], ee[3]);
                        kf[kd][m] = o.w[0];
                        kf[kd + KD / 2][m] = o.w[1];
                        kf[kd][m + 1] = o.w[2];
                        kf[kd + KD / 2][m + 1] = o.w[3];
                    }
            } else {
#pragma unroll
                for (int kd = 0; kd < KD; ++kd) {
                    const u32x4_t ee = te[kd];
                    const Words4 o = rot4_gptj(kf[kd][0], kf[kd][1], kf[kd][2], kf[kd][3], ee[0], ee[1], ee[2], ee[3]);
#pragma unroll
                    for (int m = 0; m < 4; ++m) kf[kd][m] = o.w[m];
                }
            }
        }
        f32x4_t sc4 = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kd = 0; kd < KD; ++kd)
            sc4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kf[kd]), qb[kd], sc4, 0, 0, 0);
        if (kt < kv_lo || kt + TK > kv_hi) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int key = kt + 4 * q4 + r;
                if (key < kv_lo || key >= kv_hi) sc4[r] = -INFINITY;
            }
        }
        float mx = fmaxf(fmaxf(sc4[0], sc4[1]), fmaxf(sc4[2], sc4[3]));
        mx = max_xor32(max_xor16(mx));
        if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.f) != 0) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) acc[db] *= alpha;
            m_run = m_new;
        }
        float p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            p[r] = __builtin_amdgcn_exp2f(sc4[r] - m_run);
            l_run += p[r];
        }
        const uint32_t pw[2] = {pack_bf16(p[0], p[1]), pack_bf16(p[2], p[3])};
        const bf16x4_t pb = __builtin_bit_cast(bf16x4_t, pw);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const bf16x4_t af = __builtin_bit_cast(bf16x4_t, lds_read_tr(vb + v_off[db]));
            acc[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(af, pb, acc[db], 0, 0, 0);
        }
    };

    // prologue: stages 0 .. NST-2 in flight (each issue reuses the position slot
    // the previous one read, hence the barriers)
    issue_tile(Idx<0>{}, 0);
    if constexpr (NST > 2) {
        barrier_keep_vmem();
        if (1 < n_tiles) issue_tile(Idx<1>{}, 1);
    }
    if constexpr (NST > 3) {
        barrier_keep_vmem();
        if (2 < n_tiles) issue_tile(Idx<2>{}, 2);
    }
    for (int t = 0; t < n_tiles; t += NST) {
        step(Idx<0>{}, t);
        if (t + 1 < n_tiles) step(Idx<1>{}, t + 1);
        if constexpr (NST > 2) {
            if (t + 2 < n_tiles) step(Idx<2>{}, t + 2);
        }
        if constexpr (NST > 3) {
            if (t + 3 < n_tiles) step(Idx<3>{}, t + 3);
        }
    }

    // ---- epilogue: lane l holds query column l%16 and dims 16*db + 4*(l/16) + r
    const float lt = sum_xor32(sum_xor16(l_run));
    if (!head_live || qc >= G) return;
    const int qh = kvh * G + qc;
    if (g.n_split == 1) {
        const float inv = 1.f / lt;
        uint16_t* op = static_cast<uint16_t*>(a.o) + ((size_t)g.q_row0 * a.hq + qh) * D;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const u32x2_t w = {pack_bf16(acc[db][0] * inv, acc[db][1] * inv), pack_bf16(acc[db][2] * inv, acc[db][3] * inv)};
            *reinterpret_cast<u32x2_t*>(op + db * 16 + 4 * q4) = w;
        }
    } else {
        const size_t slot = (size_t)part_base + (size_t)split * n_hg + hg;
        const int prow = wave * 16 + c16;
        float* po = a.part_o + (slot * kTileRows + prow) * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
            *reinterpret_cast<float4*>(po + db * 16 + 4 * q4) = make_float4(acc[db][0], acc[db][1], acc[db][2], acc[db][3]);
        if (q4 == 0)
            *reinterpret_cast<float2*>(a.part_ml + (slot * kTileRows + prow) * 2) = make_float2(m_run, lt);
    }
}

// decode merge: one block per (request, kMergeRows query heads), one float4 of a
// row per thread; the (max, sum) pairs and partial rows of up to 8 splits are
// loaded together before they are combined (streaming log-sum-exp)
template <int D, int HW>
__global__ void __launch_bounds__(kMergeRows * D / 4) decode_merge(const Plan plan, const Args a) {
    constexpr int TPR = D / 4;
    constexpr int U = 8;
    const int CB = dec_col_blocks(a.group), HH = HW / CB;
    const int n_hg = (a.hkv + HH - 1) / HH;
    const Group g = group_of<true>(plan, blockIdx.x);
    if (g.n_split <= 1) return;
    const int qh = ((int)blockIdx.x - g.merge_base) * kMergeRows + (int)threadIdx.x / TPR;
    const int q4 = (int)threadIdx.x % TPR;
    if (qh >= a.hq) return;
    const int kvh = qh / a.group, c = qh - kvh * a.group;
    // the decode kernel's row of this query head: its wave (KV head slot x CB +
    // column block) times 16 plus its column
    const int hg = kvh / HH, prow = ((kvh % HH) * CB + c / 16) * 16 + c % 16;
    const int L = g.tok0 + 1;
    const int n_live = min(g.n_split, (L - g.win + g.split_keys - 1) / g.split_keys);   // non-empty splits
    float M = kNegBig, den = 0.f;
    float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < n_live; s0 += U) {
        float2 ml[U];
        float4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t slot = (size_t)g.part_base + (size_t)min(s0 + u, n_live - 1) * n_hg + hg;
            ml[u] = *reinterpret_cast<const float2*>(a.part_ml + (slot * kTileRows + prow) * 2);
            v[u] = *reinterpret_cast<const float4*>(a.part_o + (slot * kTileRows + prow) * D + q4 * 4);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (s0 + u >= n_live) break;
            const float m_new = fmaxf(M, ml[u].x);
            const float c_old = __builtin_amdgcn_exp2f(M - m_new), c_new = __builtin_amdgcn_exp2f(ml[u].x - m_new);
            num.x = num.x * c_old + c_new * v[u].x;
            num.y = num.y * c_old + c_new * v[u].y;
            num.z = num.z * c_old + c_new * v[u].z;
            num.w = num.w * c_old + c_new * v[u].w;
            den = den * c_old + c_new * ml[u].y;
            M = m_new;
        }
    }
    const float inv = 1.f / den;
    uint32_t* op = reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(a.o) + ((size_t)g.q_row0 * a.hq + qh) * D + q4 * 4);
    op[0] = pack_bf16(num.x * inv, num.y * inv);
    op[1] = pack_bf16(num.z * inv, num.w * inv);
}

// ---------------------------------------------------------------------------------
// attn_f32: one wave per (query token, query head); lane holds D/64 elements.
// ---------------------------------------------------------------------------------
template <int D, int STYLE, bool ROPE, bool TABLE>
__global__ void __launch_bounds__(64) attn_f32(const Plan plan, const Args a) {
    constexpr int E = D / 64;
    constexpr int HALF = D / 2;
    const int lane = threadIdx.x;
    const int bid = blockIdx.x;
    const Group g = group_of<false>(plan, bid);
    const int li = bid - g.item_base;
    if (li >= g.n_tok * a.hq) return;
    const int toff = li / a.hq, h = li - toff * a.hq;
    const int kvh = h / a.group;
    const int t = g.tok0 + toff;

    // element e of this lane is dimension d = lane + 64 e; its pair partner and
    // frequency follow the pairing style
    auto partner_val = [&](const float* v, int e) -> float {
        if (STYLE == kNeox) {
            if (E == 2) return v[1 - e];
            return __shfl_xor(v[e], 32);
        }
        return __shfl_xor(v[e], 1);
    };
    auto rotate = [&](float* v, int32_t pos) {
        float pv[E];
#pragma unroll
        for (int e = 0; e < E; ++e) pv[e] = partner_val(v, e);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int d = lane + 64 * e;
            const int i = STYLE == kNeox ? (d % HALF) : d / 2;
            const bool first = STYLE == kNeox ? d < HALF : (d & 1) == 0;
            float c, s;
            if (TABLE && (uint32_t)pos < (uint32_t)a.rope_len) {
                const float2 cs = reinterpret_cast<const float2*>(a.rope_table)[(size_t)pos * HALF + i];
                c = cs.x; s = cs.y;
            } else {
                rope_cs(pos, a.fstep[i], c, s);
            }
            v[e] = first ? v[e] * c - pv[e] * s : v[e] * c + pv[e] * s;
        }
    };

    const float* qp = static_cast<const float*>(a.q) + ((size_t)(g.q_row0 + toff) * a.hq + h) * D;
    // element e of this lane holds kernel-layout dimension lane + 64 e of q and K
    int me[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int d = lane + 64 * e;
        me[e] = model_chunk(a.chunk_map, d >> 3) * 8 + (d & 7);
    }
    float q[E], o[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        q[e] = qp[me[e]];
        o[e] = 0.f;
    }
    if (ROPE) rotate(q, a.positions[g.pos_off + t]);
#pragma unroll
    for (int e = 0; e < E; ++e) q[e] *= a.scale_log2;

    const int32_t* btab = a.block_tables + (size_t)g.req * a.max_blocks;
    const float* kpool = static_cast<const float*>(a.k_pool);
    const float* vpool = static_cast<const float*>(a.v_pool);
    float m = kNegBig, l = 0.f;
    for (int j = g.win; j <= t; ++j) {
        const size_t base = (((size_t)btab[j >> 4] * a.hkv + kvh) * kBlock + (j & 15)) * D;
        float k[E], v[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            k[e] = kpool[base + me[e]];
            v[e] = vpool[base + lane + 64 * e];
        }
        if (ROPE) rotate(k, a.positions[g.pos_off + j]);
        float sc = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) sc += q[e] * k[e];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) sc += __shfl_xor(sc, off);
        const float m_new = fmaxf(m, sc);
        const float alpha = exp2f(m - m_new), p = exp2f(sc - m_new);
        l = l * alpha + p;
#pragma unroll
        for (int e = 0; e < E; ++e) o[e] = o[e] * alpha + p * v[e];
        m = m_new;
    }
    float* op = static_cast<float*>(a.o) + ((size_t)(g.q_row0 + toff) * a.hq + h) * D;
#pragma unroll
    for (int e = 0; e < E; ++e) op[lane + 64 * e] = o[e] / l;
}

template <int D, int STYLE, bool ROPE, bool TABLE>
hipError_t launch_attn_t(int dtype, const Plan& plan, const Args& a, hipStream_t st) {
    if (dtype == 1) {
        hipLaunchKernelGGL((attn_f32<D, STYLE, ROPE, TABLE>), dim3(plan.n_items), dim3(64), 0, st, plan, a);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((prefill_bf16<D, STYLE, ROPE, TABLE>), dim3(plan.n_items), dim3(kThreads), 0, st, plan, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (plan.n_merge > 0) {
        hipLaunchKernelGGL((merge_kernel<D>), dim3(plan.n_merge), dim3(kMergeRows * D / 8), 0, st, plan, a);
        e = hipGetLastError();
    }
    return e;
}

template <int D, int STYLE, bool ROPE, bool TABLE, int HW>
hipError_t launch_dec_w(const Plan& plan, const Args& a, hipStream_t st) {
    hipLaunchKernelGGL((decode_bf16<D, STYLE, ROPE, TABLE, HW>), dim3(plan.n_items), dim3(HW * 64), 0, st, plan, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (plan.n_merge > 0) {
        hipLaunchKernelGGL((decode_merge<D, HW>), dim3(plan.n_merge), dim3(kMergeRows * D / 4), 0, st, plan, a);
        e = hipGetLastError();
    }
    return e;
}

// decode at the workgroup width the host plan assumed (dec_waves)
template <int D, int STYLE, bool ROPE, bool TABLE>
hipError_t launch_dec_t(const Plan& plan, const Args& a, hipStream_t st) {
    if (dec_waves(D, a.hkv, a.group) == 2) return launch_dec_w<D, STYLE, ROPE, TABLE, 2>(plan, a, st);
    if (dec_waves(D, a.hkv, a.group) == 4) return launch_dec_w<D, STYLE, ROPE, TABLE, 4>(plan, a, st);
    return launch_dec_w<D, STYLE, ROPE, TABLE, dec_heads(D)>(plan, a, st);
}

template <int D, int STYLE>
hipError_t launch_dec_d(bool rope, const Plan& plan, const Args& a, hipStream_t st) {
    const bool table = a.rope_table != nullptr && a.rope_len > 0;
    if (!rope) return launch_dec_t<D, STYLE, false, false>(plan, a, st);
    return table ? launch_dec_t<D, STYLE, true, true>(plan, a, st) : launch_dec_t<D, STYLE, true, false>(plan, a, st);
}

template <int D, int STYLE>
hipError_t launch_attn_d(int dtype, bool rope, const Plan& plan, const Args& a, hipStream_t st) {
    const bool table = a.rope_table != nullptr && a.rope_len > 0;
    if (!rope) return launch_attn_t<D, STYLE, false, false>(dtype, plan, a, st);
    return table ? launch_attn_t<D, STYLE, true, true>(dtype, plan, a, st)
                 : launch_attn_t<D, STYLE, true, false>(dtype, plan, a, st);
}

}  // namespace

// ---------------------------------------------------------------------------------
// Scratch for the entry point that allocates nothing (pic_attn_decode_noalloc): a
// file-scope device array, present on every GPU the library's code is loaded on
// until the process ends.  Host code must not use the array's name as an address
// (it is a host-side stand-in): its device address is taken once per device with
// hipGetSymbolAddress, with that device current, and only that address is passed on.
// ---------------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

int scratch_region(void** ptr) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

int launch_kv_write(int dtype, int hkv, int d, void* k_pool, void* v_pool, const void* k_new, const void* v_new,
                    const int32_t* slots, int n, void* stream) {
    if (n == 0) return hipSuccess;
    const int esize = dtype == 1 ? 4 : 2;
    const int chunks_per_head = d * esize / 16;   // 4, 8, 16 or 32: a power of two
    int cph_log2 = 0;
    while ((1 << cph_log2) < chunks_per_head) ++cph_log2;
    const int per_row = hkv * chunks_per_head;
    const int threads = per_row >= 256 ? 256 : ((per_row + 63) / 64) * 64;
    hipLaunchKernelGGL(kv_write_kernel, dim3((unsigned)n), dim3(threads), 0, (hipStream_t)stream,
                       static_cast<u32x4_t*>(k_pool), static_cast<u32x4_t*>(v_pool),
                       static_cast<const u32x4_t*>(k_new), static_cast<const u32x4_t*>(v_new), slots, cph_log2, hkv);
    return hipGetLastError();
}

int launch_blocks_copy(int dtype, int hkv, int d, void* k_pool, void* v_pool, void* k_buf, void* v_buf,
                       const int32_t* block_ids, int n, bool to_pool, void* stream) {
    if (n == 0) return hipSuccess;
    const int64_t chunks = (int64_t)hkv * kBlock * d * (dtype == 1 ? 4 : 2) / 16;
    hipLaunchKernelGGL(blocks_copy_kernel, dim3((unsigned)n), dim3(256), 0, (hipStream_t)stream,
                       static_cast<u32x4_t*>(k_pool), static_cast<u32x4_t*>(v_pool), static_cast<u32x4_t*>(k_buf),
                       static_cast<u32x4_t*>(v_buf), block_ids, chunks, to_pool);
    return hipGetLastError();
}

int launch_rope_table(int dtype, int d, const RopeSteps& steps, int n_pos, float* table, void* stream) {
    const int64_t n = (int64_t)n_pos * (d / 2);
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                       static_cast<void*>(table), n_pos, d / 2, steps, dtype != 1);
    return hipGetLastError();
}

int launch_rope_rotate(int dtype, int style, int d, int rot_half, const RopeSteps& steps, const float* table, int rope_len, void* x, int n,
                       int heads, const int32_t* positions, void* stream) {
    const int64_t n_pairs = (int64_t)n * heads * (d / 2);
    if (n_pairs == 0) return hipSuccess;
    const dim3 grid((unsigned)((n_pairs + 255) / 256));
    const void* t = table;
    hipStream_t st = (hipStream_t)stream;
    if (dtype == 1) {
        if (style == kNeox)
            hipLaunchKernelGGL((rope_rotate_kernel<float, 0>), grid, dim3(256), 0, st, static_cast<float*>(x),
                               n_pairs, heads, d, rot_half, steps, positions, t, rope_len);
        else
            hipLaunchKernelGGL((rope_rotate_kernel<float, 1>), grid, dim3(256), 0, st, static_cast<float*>(x),
                               n_pairs, heads, d, rot_half, steps, positions, t, rope_len);
    } else {
        if (style == kNeox)
            hipLaunchKernelGGL((rope_rotate_kernel<__bf16, 0>), grid, dim3(256), 0, st, static_cast<__bf16*>(x),
                               n_pairs, heads, d, rot_half, steps, positions, t, rope_len);
        else
            hipLaunchKernelGGL((rope_rotate_kernel<__bf16, 1>), grid, dim3(256), 0, st, static_cast<__bf16*>(x),
                               n_pairs, heads, d, rot_half, steps, positions, t, rope_len);
    }
    return hipGetLastError();
}

int launch_plan_upload(const PlanUpload& up, void* stream) {
    if (up.n <= 0) return hipSuccess;
    hipLaunchKernelGGL(plan_upload_kernel, dim3((unsigned)up.n), dim3(256), 0, (hipStream_t)stream, up);
    return hipGetLastError();
}

int launch_decode(int style, int d, bool rope, const Plan& plan, const Args& args, void* stream) {
    if (plan.n_items == 0) return hipSuccess;
    hipStream_t st = (hipStream_t)stream;
    if (d == 64)
        return style == kNeox ? launch_dec_d<64, 0>(rope, plan, args, st) : launch_dec_d<64, 1>(rope, plan, args, st);
    return style == kNeox ? launch_dec_d<128, 0>(rope, plan, args, st) : launch_dec_d<128, 1>(rope, plan, args, st);
}

int launch_attention(int dtype, int style, int d, bool rope, const Plan& plan, const Args& args, void* stream) {
    if (plan.n_items == 0) return hipSuccess;
    hipStream_t st = (hipStream_t)stream;
    if (d == 64)
        return style == kNeox ? launch_attn_d<64, 0>(dtype, rope, plan, args, st)
                              : launch_attn_d<64, 1>(dtype, rope, plan, args, st);
    return style == kNeox ? launch_attn_d<128, 0>(dtype, rope, plan, args, st)
                          : launch_attn_d<128, 1>(dtype, rope, plan, args, st);
}

}  // namespace pic
