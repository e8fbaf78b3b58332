// Host side of the span cache: SHA-256, the block-hash rule of eq. (1)
// (Sec. 3.1.1), span boundaries from cache hits, and a hash -> block map.
// Declared in include/pic_cache.h.  Nothing here touches the GPU.
#include <algorithm>
#include <array>
#include <cstring>
#include <unordered_map>

#include "pic_cache.h"
#include "pic_internal.h"

namespace {

// ---------------------------------------------------------------------------
// SHA-256 (FIPS 180-4, Sec. 5.1.1 padding, 6.2 computation).  The round
// constants are the first 32 fractional bits of the cube roots of the first 64
// primes and the initial state those of the square roots of the first 8.
// ---------------------------------------------------------------------------
constexpr uint32_t kRound[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u, 0xab1c5ed5u,
    0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u,
    0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u,
    0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u,
    0xa2bfe8a1u, 0xa81a664bu, 0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u,
};
constexpr uint32_t kInit[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                               0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

inline uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

class Sha256 {
public:
    Sha256() { std::memcpy(h_, kInit, sizeof h_); }

    void update(const void* data, size_t n) {
        const uint8_t* p = static_cast<const uint8_t*>(data);
        total_ += n;
        if (fill_ > 0) {
            const size_t take = std::min(n, size_t(64) - fill_);
            std::memcpy(buf_ + fill_, p, take);
            fill_ += take;
            p += take;
            n -= take;
            if (fill_ < 64) return;
            compress(buf_);
            fill_ = 0;
        }
        for (; n >= 64; p += 64, n -= 64) compress(p);
        std::memcpy(buf_, p, n);
        fill_ = n;
    }

    void final(uint8_t out[32]) {
        // message || 0x80 || zeros || 64-bit big-endian bit length, to a multiple of 64 bytes
        const uint64_t bits = uint64_t(total_) * 8;
        const uint8_t one = 0x80;
        uint8_t zeros[64] = {};
        update(&one, 1);
        update(zeros, (fill_ <= 56 ? 56 : 120) - fill_);
        uint8_t len[8];
        for (int i = 0; i < 8; ++i) len[i] = uint8_t(bits >> (56 - 8 * i));
        update(len, 8);
        for (int i = 0; i < 8; ++i)
            for (int j = 0; j < 4; ++j) out[4 * i + j] = uint8_t(h_[i] >> (24 - 8 * j));
    }

private:
    void compress(const uint8_t* blk) {
        uint32_t w[64];
        for (int t = 0; t < 16; ++t)
            w[t] = uint32_t(blk[4 * t]) << 24 | uint32_t(blk[4 * t + 1]) << 16 | uint32_t(blk[4 * t + 2]) << 8 |
                   uint32_t(blk[4 * t + 3]);
        for (int t = 16; t < 64; ++t) {
            const uint32_t s0 = rotr(w[t - 15], 7) ^ rotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
            const uint32_t s1 = rotr(w[t - 2], 17) ^ rotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
            w[t] = w[t - 16] + s0 + w[t - 7] + s1;
        }
        uint32_t a = h_[0], b = h_[1], c = h_[2], d = h_[3], e = h_[4], f = h_[5], g = h_[6], h = h_[7];
        for (int t = 0; t < 64; ++t) {
            const uint32_t t1 = h + (rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25)) + ((e & f) ^ (~e & g)) + kRound[t] + w[t];
            const uint32_t t2 = (rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22)) + ((a & b) ^ (a & c) ^ (b & c));
            h = g;
            g = f;
            f = e;
            e = d + t1;
            d = c;
            c = b;
            b = a;
            a = t1 + t2;
        }
        h_[0] += a; h_[1] += b; h_[2] += c; h_[3] += d;
        h_[4] += e; h_[5] += f; h_[6] += g; h_[7] += h;
    }

    uint32_t h_[8];
    uint8_t buf_[64];
    size_t fill_ = 0;
    size_t total_ = 0;
};

// block tokens as the little-endian int32 bytes H consumes
void hash_tokens(Sha256& s, const int32_t* tok, int n) {
    uint8_t bytes[4 * pic::kBlock];
    for (int t = 0; t < n; ++t) {
        const uint32_t u = uint32_t(tok[t]);
        for (int j = 0; j < 4; ++j) bytes[4 * t + j] = uint8_t(u >> (8 * j));
    }
    s.update(bytes, size_t(4) * n);
}

using Digest = std::array<uint8_t, 32>;

struct DigestHash {
    size_t operator()(const Digest& d) const {
        uint64_t v;  // the digest is uniformly distributed: any 8 bytes make a good key
        std::memcpy(&v, d.data(), sizeof v);
        return size_t(v);
    }
};

}  // namespace

struct pic_block_cache {
    std::unordered_map<Digest, int32_t, DigestHash> map;
};

extern "C" {

pic_status pic_sha256(const void* data, size_t bytes, uint8_t* out) {
    if (out == nullptr || (data == nullptr && bytes > 0)) return pic::host_fail(PIC_EINVAL, "pic_sha256: NULL pointer");
    Sha256 s;
    if (bytes > 0) s.update(data, bytes);
    s.final(out);
    return PIC_OK;
}

pic_status pic_block_hashes(const int32_t* tokens, int32_t n_tokens, int32_t ssep_token, int32_t pdep_token,
                            const uint8_t* seed, uint8_t* out) {
    if (n_tokens < 0) return pic::host_fail(PIC_EINVAL, "pic_block_hashes: n_tokens < 0");
    if (ssep_token == pdep_token) return pic::host_fail(PIC_EINVAL, "pic_block_hashes: ssep_token == pdep_token");
    const int nb = n_tokens / pic::kBlock;
    if (seed == nullptr || (n_tokens > 0 && tokens == nullptr) || (nb > 0 && out == nullptr))
        return pic::host_fail(PIC_EINVAL, "pic_block_hashes: NULL pointer");
    // `prefix` absorbs h_0 and every token so far, so that the PDEP case, the
    // hash of h_0 followed by all tokens up to the end of the block, costs one
    // copy of the running state instead of rehashing the prefix.
    Sha256 prefix;
    prefix.update(seed, 32);
    const uint8_t* prev = seed;
    for (int b = 0; b < nb; ++b) {
        const int32_t* x = tokens + size_t(b) * pic::kBlock;
        uint8_t* h = out + size_t(b) * 32;
        hash_tokens(prefix, x, pic::kBlock);
        if (x[0] == pdep_token) {
            Sha256 s = prefix;
            s.final(h);
        } else {
            Sha256 s;
            s.update(x[0] == ssep_token ? seed : prev, 32);
            hash_tokens(s, x, pic::kBlock);
            s.final(h);
        }
        prev = h;
    }
    return PIC_OK;
}

pic_status pic_spans_from_blocks(const int32_t* tokens, int32_t n_tokens, int32_t ssep_token, int32_t pdep_token,
                                 const uint8_t* hit, int32_t* span_start, int32_t* span_flags, int32_t capacity,
                                 int32_t* n_spans) {
    if (n_tokens <= 0) return pic::host_fail(PIC_EINVAL, "pic_spans_from_blocks: n_tokens must be positive");
    if (ssep_token == pdep_token) return pic::host_fail(PIC_EINVAL, "pic_spans_from_blocks: ssep_token == pdep_token");
    const int full = n_tokens / pic::kBlock;
    const int nb = (n_tokens + pic::kBlock - 1) / pic::kBlock;
    if (tokens == nullptr || n_spans == nullptr || (full > 0 && hit == nullptr) ||
        (capacity > 0 && (span_start == nullptr || span_flags == nullptr)))
        return pic::host_fail(PIC_EINVAL, "pic_spans_from_blocks: NULL pointer");
    int count = 0;
    bool prev_cached = false;
    for (int b = 0; b < nb; ++b) {
        const int32_t first = tokens[size_t(b) * pic::kBlock];
        const int32_t marker = first == ssep_token ? PIC_SSEP : first == pdep_token ? PIC_PDEP : 0;
        const bool cached = b < full && hit[b] != 0;
        // A marker opens a span with its own window.  Otherwise a change between
        // cached and computed blocks opens an unflagged span, which keeps the
        // window of the span before it, so the attention mask is that of the
        // marker structure alone whatever hits.
        if (b == 0 || marker != 0 || cached != prev_cached) {
            if (count < capacity) {
                span_start[count] = b * pic::kBlock;
                span_flags[count] = marker | (cached ? 0 : PIC_QUERY);
            }
            ++count;
        }
        prev_cached = cached;
    }
    *n_spans = count;
    if (count > capacity) return pic::host_fail(PIC_EINVAL, "pic_spans_from_blocks: capacity < number of spans");
    return PIC_OK;
}

pic_status pic_block_cache_create(pic_block_cache** cache) {
    if (cache == nullptr) return pic::host_fail(PIC_EINVAL, "pic_block_cache_create: NULL pointer");
    *cache = new pic_block_cache();
    return PIC_OK;
}

pic_status pic_block_cache_destroy(pic_block_cache* cache) {
    delete cache;
    return PIC_OK;
}

pic_status pic_block_cache_lookup(const pic_block_cache* cache, const uint8_t* hashes, int32_t n, int32_t* block_ids,
                                  int32_t* n_hits) {
    if (cache == nullptr || n < 0 || (n > 0 && (hashes == nullptr || block_ids == nullptr)))
        return pic::host_fail(PIC_EINVAL, "pic_block_cache_lookup: bad argument");
    int32_t hits = 0;
    Digest d;
    for (int i = 0; i < n; ++i) {
        std::memcpy(d.data(), hashes + size_t(i) * 32, 32);
        const auto it = cache->map.find(d);
        block_ids[i] = it == cache->map.end() ? -1 : it->second;
        hits += it != cache->map.end();
    }
    if (n_hits != nullptr) *n_hits = hits;
    return PIC_OK;
}

pic_status pic_block_cache_insert(pic_block_cache* cache, const uint8_t* hashes, const int32_t* block_ids,
                                  int32_t n) {
    if (cache == nullptr || n < 0 || (n > 0 && (hashes == nullptr || block_ids == nullptr)))
        return pic::host_fail(PIC_EINVAL, "pic_block_cache_insert: bad argument");
    Digest d;
    for (int i = 0; i < n; ++i) {
        if (block_ids[i] < 0) continue;
        std::memcpy(d.data(), hashes + size_t(i) * 32, 32);
        cache->map.emplace(d, block_ids[i]);
    }
    return PIC_OK;
}

pic_status pic_block_cache_erase(pic_block_cache* cache, const uint8_t* hashes, int32_t n) {
    if (cache == nullptr || n < 0 || (n > 0 && hashes == nullptr))
        return pic::host_fail(PIC_EINVAL, "pic_block_cache_erase: bad argument");
    Digest d;
    for (int i = 0; i < n; ++i) {
        std::memcpy(d.data(), hashes + size_t(i) * 32, 32);
        cache->map.erase(d);
    }
    return PIC_OK;
}

pic_status pic_block_cache_size(const pic_block_cache* cache, int32_t* size) {
    if (cache == nullptr || size == nullptr) return pic::host_fail(PIC_EINVAL, "pic_block_cache_size: NULL pointer");
    *size = int32_t(cache->map.size());
    return PIC_OK;
}

}  // extern "C"
