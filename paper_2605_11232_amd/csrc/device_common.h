// Device-side helpers shared by the HIP kernels of libpa (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBlock = 16;                     // tokens per KV block
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 zero16() { return u32x4{0u, 0u, 0u, 0u}; }

// Keep only the first `keep` (0..8) bf16 lanes of a 16-byte vector.
__device__ __forceinline__ u32x4 keep_bf16(u32x4 v, int keep) {
  u32x4 r;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int e0 = 2 * k;
    uint32_t m = (e0 < keep ? 0x0000FFFFu : 0u) | (e0 + 1 < keep ? 0xFFFF0000u : 0u);
    r[k] = v[k] & m;
  }
  return r;
}

// 32x32x16 bf16 MFMA: C[32x32] += A[32x16] * B[16x32].  Lane l holds A row
// l % 32 and B column l % 32, k elements 8 * (l / 32) .. + 7; C column l % 32,
// rows 8 * (e / 4) + 4 * (l / 32) + e % 4 for element e.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// 16x16x32 bf16 MFMA: lane l holds A row l % 16 and B column l % 16, k elements
// 8 * (l / 16) .. + 7; C column l % 16, rows 4 * (l / 16) + e.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the hardware transcendental unit (v_exp_f32) without the library's
// denormal-range fix-up: results below 2^-126 flush to zero, which only
// drops probabilities that are negligible against the row maximum (>= 1).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }

// A wavefront's view of 64 consecutive entries of a block-table row, one per
// lane, with the next 64 loaded one window ahead: block ids are then read with
// v_readlane (no scalar-memory wait inside the key loop).
struct BlockWindow {
  const int32_t* row;
  int last;        // table index of the last block in use; later entries read it again
  int num_blocks;  // ids are clamped to [0, num_blocks) when fetched
  int base;        // first block index held in `cur`
  int cur, next;

  __device__ __forceinline__ int fetch(int first) const {
    const int j = first + (threadIdx.x & 63);
    const int id = row[j < last ? j : last];
    return id < 0 ? 0 : (id >= num_blocks ? num_blocks - 1 : id);
  }
  __device__ __forceinline__ void init(const int32_t* r, int last_block, int nblocks, int first_block) {
    row = r;
    last = last_block;
    num_blocks = nblocks;
    base = first_block;
    cur = fetch(base);
    next = fetch(base + 64);
  }
  // Make logical blocks jb .. jb + n - 1 readable with at() (wave-uniform;
  // jb >= base, non-decreasing; the n blocks must not straddle a window, which
  // holds when the caller steps through its blocks n at a time from the first
  // block it passed to init).
  __device__ __forceinline__ void seek(int jb) {
    while (jb - base >= 64) {
      base += 64;
      cur = next;
      next = fetch(base + 64);
    }
  }
  __device__ __forceinline__ int at(int jb) const {
    return __builtin_amdgcn_readlane(cur, jb - base);
  }
  // Block id of logical block jb (wave-uniform, jb >= base, non-decreasing).
  __device__ __forceinline__ int get(int jb) {
    seek(jb);
    return at(jb);
  }
};

// A wavefront's view of at most 64 consecutive entries of a block-table row,
// one per lane, loaded once (items that never span more than 64 blocks): no
// table load inside the key loop, so the loop's memory waits only concern
// its key and value loads.
struct BlockSpan {
  int base;  // first block index held
  int ids;
  __device__ __forceinline__ void init(const int32_t* row, int max_blocks, int first_block) {
    base = first_block;
    const int j = first_block + (threadIdx.x & 63);
    ids = row[j < max_blocks ? j : max_blocks - 1];
  }
  // Block id of logical block jb, base <= jb < base + 64 (wave-uniform).
  __device__ __forceinline__ int get(int jb) const {
    return __builtin_amdgcn_readlane(ids, (jb - base) & 63);
  }
};

// Key cache layout.  One (block, kv-head) of keys is [D/32][16][32]: for each
// group of 32 head dimensions, the block's 16 token slots of 32 dims each.
// A slot's position inside a group is its offset with bits 2 and 3 swapped,
// so the eight keys a decode MFMA tile needs from one block (offsets
// 0-3 and 8-11, or 4-7 and 12-15) are 256 contiguous bytes of each group.
constexpr int kKeyGroup = 32;
__host__ __device__ constexpr int key_slot_pos(int off) {
  return (off & ~12) | ((off & 4) << 1) | ((off & 8) >> 1);
}
// Element offset of (token offset off, dim d) inside one (block, kv-head).
__host__ __device__ constexpr int key_elem(int off, int d) {
  return (d / kKeyGroup) * (kBlock * kKeyGroup) + key_slot_pos(off) * kKeyGroup + d % kKeyGroup;
}

__device__ __forceinline__ int clamp_block(int b, int num_blocks) {
  return b < 0 ? 0 : (b >= num_blocks ? num_blocks - 1 : b);
}

}  // namespace dev
}  // namespace pa
