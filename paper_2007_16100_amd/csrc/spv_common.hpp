// spv_common.hpp -- device helpers shared by the HIP kernels of libspv.so:
// packed voxel keys, the open-addressing hash, 16-bit storage conversions,
// MFMA operand types, the device status word and the workspace arena.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/spv.h"

namespace spv {

// ---------------------------------------------------------------------------
// packed voxel keys: b:16 | (x + 2^15):16 | (y + 2^15):16 | (z + 2^15):16.
// The packing is monotone, so key order is (b, x, y, z) lexicographic order.
// Batch 65535 is reserved, which makes all-ones the empty-slot sentinel.
// ---------------------------------------------------------------------------
constexpr uint64_t kEmpty = ~0ull;
constexpr int kCoordMin = -32767;
constexpr int kCoordMax = 32766;
constexpr int kBatchMax = 65534;
__host__ __device__ inline bool in_key_range(int c) { return c >= kCoordMin && c <= kCoordMax; }

__host__ __device__ inline uint64_t pack_key(int b, int x, int y, int z) {
    return ((uint64_t)(uint32_t)b << 48) | ((uint64_t)(uint32_t)(x + 32768) << 32) |
           ((uint64_t)(uint32_t)(y + 32768) << 16) | (uint64_t)(uint32_t)(z + 32768);
}
__host__ __device__ inline int key_b(uint64_t k) { return (int)(k >> 48); }
__host__ __device__ inline int key_x(uint64_t k) { return (int)((k >> 32) & 0xFFFF) - 32768; }
__host__ __device__ inline int key_y(uint64_t k) { return (int)((k >> 16) & 0xFFFF) - 32768; }
__host__ __device__ inline int key_z(uint64_t k) { return (int)(k & 0xFFFF) - 32768; }

// ---------------------------------------------------------------------------
// device status word (bit flags); the host reports the most severe one
// ---------------------------------------------------------------------------
enum : uint32_t {
    kFlagNonfinite = 1u << 0,
    kFlagRange = 1u << 1,
    kFlagCapacity = 1u << 2,
    kFlagDuplicate = 1u << 3,  // repeated coordinate where distinct ones are required
    kFlagTableFull = 1u << 4,
    kFlagUnsorted = 1u << 5,   // a kernel-map offset group not sorted by output row
    kFlagInternal = 1u << 6,   // a kernel gave up waiting on another (a runtime fault, not an input error)
};

// Workspace header: first 256 bytes of every workspace.
struct alignas(256) Header {
    uint32_t status;
    uint32_t pad;
    int64_t m;              // unique voxels inserted by the voxelization
    int64_t aux[4];         // [0]: voxels the scatter-mean sums with a whole workgroup
};

__device__ inline void raise_flag(Header* h, uint32_t f) { atomicOr(&h->status, f); }

// ---------------------------------------------------------------------------
// open-addressing hash with linear probing over 64-bit keys.  A probe sequence
// starts at the first slot of a 4-slot bucket and continues linearly, wrapping
// at the end of the table; lookups read one whole bucket (4 keys + 4 values)
// per round, so almost every lookup costs a single memory round trip.  A
// bucket is one 64-byte block -- its 4 keys, its 4 values, 16 bytes unused --
// so a probe touches a single cache line.
// ---------------------------------------------------------------------------
typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
typedef int i32x4v __attribute__((ext_vector_type(4)));

__host__ __device__ inline uint32_t hash_slot(uint64_t k, uint32_t mask) {
    // murmur3 64-bit finalizer, scaled to a bucket's first slot
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdull;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ull;
    k ^= k >> 33;
    return ((uint32_t)k << 2) & mask;
}

constexpr uint32_t kNoSlot = 0xFFFFFFFFu;  // "no table slot"

struct Table {
    uint64_t* keys;  // bucket-major storage, 16 bytes per slot, 256-byte aligned (see table_words)
    uint32_t mask;   // capacity - 1 (capacity is a power of two, >= 4)
};
// 64-bit words of a table of S slots: S / 4 buckets of 8 words
__host__ __device__ inline size_t table_words(uint32_t S) { return (size_t)2 * S; }
// the key and the value of slot s
__device__ inline uint64_t* slot_key(Table t, uint32_t s) { return t.keys + 8 * (size_t)(s >> 2) + (s & 3); }
__device__ inline int32_t* slot_val(Table t, uint32_t s) {
    return (int32_t*)(t.keys + 8 * (size_t)(s >> 2) + 4) + (s & 3);
}

// Insert; returns 1 if this call created the entry, 0 if the key was present,
// -1 if the table is full.  *slot receives the entry's slot.  Slots are claimed
// strictly in probe order, so a lookup may stop at the first empty slot.
// Every probe step is one compare-and-swap (empty -> key): on a table this
// sparse the first slot is usually empty or already holds the key, and a CAS
// settles both in one round trip, where a load first would take two.
__device__ inline int table_insert(Table t, uint64_t key, uint32_t* slot) {
    uint32_t s = hash_slot(key, t.mask);
    for (uint32_t i = 0; i <= t.mask; ++i) {
        const uint64_t prev = atomicCAS((unsigned long long*)slot_key(t, s), (unsigned long long)kEmpty,
                                        (unsigned long long)key);
        if (prev == kEmpty) {
            *slot = s;
            return 1;
        }
        if (prev == key) {
            *slot = s;
            return 0;
        }
        s = (s + 1) & t.mask;
    }
    return -1;
}

// One bucket of a probe: keys s..s+3 (s a multiple of 4) and their values.
struct Bucket {
    u64x2 k01, k23;
    i32x4v v;
};
__device__ inline Bucket load_bucket(Table t, uint32_t s) {
    const uint64_t* q = t.keys + 8 * (size_t)(s >> 2);
    Bucket b;
    b.k01 = *(const u64x2*)q;
    b.k23 = *(const u64x2*)(q + 2);
    b.v = *(const i32x4v*)(q + 4);
    return b;
}
// settle a lookup from one bucket: 1 = found (*pos = slot offset 0..3),
// 0 = absent (an empty slot came first), -1 = continue with the next bucket
__device__ inline int bucket_match(const Bucket& b, uint64_t key, int* pos) {
    const uint64_t k[4] = {b.k01.x, b.k01.y, b.k23.x, b.k23.y};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (k[e] == key) {
            *pos = e;
            return 1;
        }
        if (k[e] == kEmpty) return 0;
    }
    return -1;
}
__device__ inline int32_t bucket_val(const Bucket& b, int e) {
    return e == 0 ? b.v.x : e == 1 ? b.v.y : e == 2 ? b.v.z : b.v.w;
}

// slot of a present key, -1 if absent; the probe starts at bucket slot s
__device__ inline int64_t table_slot_from(Table t, uint64_t key, uint32_t s) {
    for (uint32_t i = 0; i <= t.mask; i += 4) {
        const Bucket b = load_bucket(t, s);
        int e = 0;
        const int r = bucket_match(b, key, &e);
        if (r > 0) return (int64_t)(s + e);
        if (r == 0) return -1;
        s = (s + 4) & t.mask;
    }
    return -1;
}

// Lookup after the table is complete (a later kernel); -1 if absent.
__device__ inline int32_t table_find(Table t, uint64_t key) {
    uint32_t s = hash_slot(key, t.mask);
    for (uint32_t i = 0; i <= t.mask; i += 4) {
        const Bucket b = load_bucket(t, s);
        int e = 0;
        const int r = bucket_match(b, key, &e);
        if (r > 0) return bucket_val(b, e);
        if (r == 0) return -1;
        s = (s + 4) & t.mask;
    }
    return -1;
}

// slot of a present key (used to set values); -1 if absent
__device__ inline int64_t table_slot(Table t, uint64_t key) { return table_slot_from(t, key, hash_slot(key, t.mask)); }

// NP lookups whose first buckets are read together, keys only (two 16-byte
// loads per probe, one round trip for all of them); the values of the keys
// found there are read next, one 4-byte load each.  A probe settles in its
// first bucket when the key is there or a slot of the bucket is empty (an
// insert would have stopped at that slot); the rare other one continues
// bucket by bucket on its own.  Inactive entries (act[p] false) read bucket 0
// and return -1.
template <int NP>
__device__ inline void table_find_n(Table t, const uint64_t (&key)[NP], const bool (&act)[NP], int32_t (&res)[NP]) {
    uint32_t s[NP];
    u64x2 a[NP], b[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        s[p] = act[p] ? hash_slot(key[p], t.mask) : 0u;
        const uint64_t* q = t.keys + 8 * (size_t)(s[p] >> 2);
        a[p] = *(const u64x2*)q;
        b[p] = *(const u64x2*)(q + 2);
    }
    int e[NP];  // slot of the key in the bucket (0..3), -1 absent, -2 continue
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        const uint64_t k4[4] = {a[p].x, a[p].y, b[p].x, b[p].y};
        bool empty = false;
        e[p] = -1;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (k4[u] == key[p]) e[p] = u;  // a key is stored at most once
            empty = empty || k4[u] == kEmpty;
        }
        if (!act[p]) e[p] = -1;
        else if (e[p] < 0 && !empty) e[p] = -2;
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        res[p] = -1;
        if (e[p] >= 0) {
            res[p] = *((const int32_t*)(t.keys + 8 * (size_t)(s[p] >> 2) + 4) + e[p]);
        } else if (e[p] == -2) {
            const int64_t sl = table_slot_from(t, key[p], (s[p] + 4) & t.mask);
            res[p] = sl >= 0 ? *slot_val(t, (uint32_t)sl) : -1;
        }
    }
}

// a table of S slots (a power of two, >= 4) carved from an arena
template <class A>
inline Table take_table(A& a, uint32_t S) {
    return Table{a.template take<uint64_t>(table_words(S)), S - 1};
}

inline uint32_t table_capacity(int64_t max_keys) {
    uint64_t c = 1024;
    while (c < (uint64_t)(2 * max_keys)) c <<= 1;
    return (uint32_t)c;
}

// ---------------------------------------------------------------------------
// 16-bit storage
// ---------------------------------------------------------------------------
__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ inline uint16_t f32_to_bf16(float f) {  // round to nearest even
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ inline float f16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
__device__ inline uint16_t f32_to_f16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

template <int DT>
__device__ inline float ld_feat(const void* p, int64_t i) {
    if constexpr (DT == SPV_F32) return ((const float*)p)[i];
    else if constexpr (DT == SPV_BF16) return bf16_to_f32(((const uint16_t*)p)[i]);
    else return f16_to_f32(((const uint16_t*)p)[i]);
}
template <int DT>
__device__ inline void st_feat(void* p, int64_t i, float v) {
    if constexpr (DT == SPV_F32) ((float*)p)[i] = v;
    else if constexpr (DT == SPV_BF16) ((uint16_t*)p)[i] = f32_to_bf16(v);
    else ((uint16_t*)p)[i] = f32_to_f16(v);
}
template <int DT>
__device__ inline uint16_t to16(float v) {
    if constexpr (DT == SPV_BF16) return f32_to_bf16(v);
    else return f32_to_f16(v);
}
// fp64 -> fp32 rounding to odd: a following round-to-nearest-even to a format
// with at most 22 fraction bits then rounds the fp64 value exactly once
__device__ inline float f64_to_f32_odd(double d) {
    float f = __double2float_rz(d);
    if ((double)f != d) f = __uint_as_float(__float_as_uint(f) | 1u);
    return f;
}
template <int DT>
__device__ inline float from16(uint32_t h) {
    if constexpr (DT == SPV_BF16) return bf16_to_f32((uint16_t)h);
    else return f16_to_f32((uint16_t)h);
}

// ---------------------------------------------------------------------------
// MFMA operand types (gfx950: v_mfma_f32_16x16x32_{bf16,f16})
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int DT>
__device__ inline f32x4 mfma16x16x32(uint4 a, uint4 b, f32x4 c) {
    if constexpr (DT == SPV_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                      0, 0);
}

// ---------------------------------------------------------------------------
// host-side workspace arena: sequential 256-byte aligned carving
// ---------------------------------------------------------------------------
struct Arena {
    char* base;
    size_t cap;
    size_t used = 0;
    Arena(void* b, size_t c) : base((char*)b), cap(c) {}
    template <class T>
    T* take(size_t count) {
        size_t off = (used + 255) & ~(size_t)255;
        used = off + count * sizeof(T);
        return (base && used <= cap) ? (T*)(base + off) : nullptr;
    }
    bool ok() const { return used <= cap; }
};

inline unsigned blocks_for(int64_t n, int per_block) {
    int64_t b = (n + per_block - 1) / per_block;
    return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace spv
