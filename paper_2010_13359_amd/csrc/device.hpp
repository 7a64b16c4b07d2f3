// Device helpers for the DQGAN compression kernels (gfx950 / CDNA4).
//
// Lane layout used by every element-wise kernel: a lane owns one "quad" of
// four consecutive elements (one 128-bit load per row), a 64-lane wavefront
// covers 256 consecutive elements, a 256-thread workgroup covers 1024.  Row
// strides are multiples of 1024, so a workgroup never straddles a row end.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dq {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;          // threads per workgroup
constexpr int kQuadsPerBlock = 256;  // one quad per thread
constexpr int kElemsPerBlock = 1024;

// Streaming 128-bit accesses.  The gradient, residual and evaluation-point
// matrices are touched once per pass, so they bypass cache retention.
__device__ __forceinline__ f32x4 ld_stream(const float *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
}
__device__ __forceinline__ void st_stream(float *p, f32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
}
__device__ __forceinline__ f32x4 ld4(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }
__device__ __forceinline__ void st4(float *p, f32x4 v) { *reinterpret_cast<f32x4 *>(p) = v; }

// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32->64-bit
// products (multipliers 0xD2511F53, 0xCD9E8D57) mixed with the key, which
// advances by the Weyl constants (0x9E3779B9, 0xBB67AE85) after every round.
__device__ __forceinline__ u32x4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                               uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t a = static_cast<uint64_t>(c0) * 0xD2511F53u;
        const uint64_t b = static_cast<uint64_t>(c2) * 0xCD9E8D57u;
        const uint32_t n0 = static_cast<uint32_t>(b >> 32) ^ c1 ^ k0;
        const uint32_t n2 = static_cast<uint32_t>(a >> 32) ^ c3 ^ k1;
        c1 = static_cast<uint32_t>(b);
        c3 = static_cast<uint32_t>(a);
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    u32x4 out;
    out.x = c0;
    out.y = c1;
    out.z = c2;
    out.w = c3;
    return out;
}

// OR of a 32-bit value over each aligned group of 8 lanes, via DPP: two quad
// permutations (xor 1, xor 2) then a row shift by 4.  The full OR is valid in
// lanes 4..7 of each group of 8 (lane & 7 == 4 is the writer).
__device__ __forceinline__ uint32_t or_reduce8_to_lane4(uint32_t x) {
    x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0xB1, 0xF, 0xF, true));
    x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x4E, 0xF, 0xF, true));
    x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x114, 0xF, 0xF, true));
    return x;
}

// Stores of a packed field plane, one quad per lane.  The fields of
// consecutive lanes are gathered with DPP: lane pairs form a word (quad_perm
// 1,0,3,2); lane 8j (4-bit fields) or 4j (8-bit fields) collects the next
// words with row shifts and writes 16 bytes with one non-temporal store.
// Every lane of the wave must be active; `row` is 16-byte aligned; lane 8j /
// 4j holds quad q with q % 8 == 0 / q % 4 == 0.
//
// 4-bit fields (16 bits per lane): sub-dword stores of the same bytes made
// the fused pass 9 % slower than its compute-free access pattern; the
// gathered streaming store runs at the pattern's rate.
__device__ __forceinline__ void store_fields16(uint32_t *__restrict__ row, int64_t q, uint32_t h) {
    const uint32_t hp = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(h), 0xB1, 0xF, 0xF, true));
    const uint32_t wv = (h & 0xFFFFu) | (hp << 16);
    u32x4 v;
    v.x = wv;
    v.y = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(wv), 0x102, 0xF, 0xF, true));
    v.z = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(wv), 0x104, 0xF, 0xF, true));
    v.w = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(wv), 0x106, 0xF, 0xF, true));
    if ((q & 7) == 0) __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(row + (q >> 1)));
}

// 8-bit fields (32 bits per lane).  STREAM: the plane is larger than the
// 256 MB Infinity Cache, where the gathered streaming store is 4-5 % faster
// (32 workers x 33.5M elements, a 1.07 GB plane); a smaller plane keeps one
// cache-allocating 32-bit store per lane (streaming made the 0.1 GB planes of
// 16 workers x 6.3M elements 5 % slower: the cache defers their write-back
// past the pass).
template <bool STREAM>
__device__ __forceinline__ void store_fields32(uint32_t *__restrict__ row, int64_t q, uint32_t w) {
    if (!STREAM) {
        row[q] = w;
        return;
    }
    u32x4 v;
    v.x = w;
    v.y = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(w), 0x101, 0xF, 0xF, true));
    v.z = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(w), 0x102, 0xF, 0xF, true));
    v.w = static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(w), 0x103, 0xF, 0xF, true));
    if ((q & 3) == 0) __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(row + q));
}

// Segment of element i, scanning forward from segment j (offsets ascending).
__device__ __forceinline__ int seg_from(const int64_t *__restrict__ off, int j, int64_t i) {
    while (off[j + 1] <= i) ++j;
    return j;
}

// binary32 operations spelled out (the library is built with
// -ffp-contract=off; these keep each product and sum a separate rounding).
__device__ __forceinline__ float mul_rn(float a, float b) { return __fmul_rn(a, b); }
__device__ __forceinline__ float add_rn(float a, float b) { return __fadd_rn(a, b); }
__device__ __forceinline__ float sub_rn(float a, float b) { return __fsub_rn(a, b); }

__device__ __forceinline__ float elem(const f32x4 &v, int c) {
    return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set_elem(f32x4 &v, int c, float x) {
    if (c == 0) v.x = x;
    else if (c == 1) v.y = x;
    else if (c == 2) v.z = x;
    else v.w = x;
}
__device__ __forceinline__ uint32_t elem(const u32x4 &v, int c) {
    return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
}

}  // namespace dq
