// KV append: scatter the keys/values of new tokens into their cache slots.
//
// Paper: Section 2 (PagedAttention keeps each token's keys and values in the
// block and offset its block table maps it to).  Keys go to the grouped
// layout of device_common.h ([block][head][dim / 32][slot position][32]):
// each token-head row is copied with 16-byte loads and stores, as 64-byte
// (bf16) or 128-byte (fp32) runs per 32-dim group.  Values are stored transposed per block
// ([block][head][dim][offset]) so attention reads keys contiguously in the PV
// product; a workgroup stages 16 consecutive tokens of one head in LDS and
// writes each dimension's 16 offsets as neighbouring elements, so tokens that
// fill one block produce full 32-byte (bf16) or 64-byte (fp32) runs.
#include "device_common.h"

namespace pa {
namespace dev {
namespace {

template <typename T, int D>
__global__ __launch_bounds__(256) void kv_append_kernel(const T* __restrict__ k_new,
                                                        const T* __restrict__ v_new,
                                                        const int32_t* __restrict__ slots,
                                                        int32_t n_tokens, T* __restrict__ kc,
                                                        T* __restrict__ vc, int32_t num_blocks,
                                                        int32_t hkv) {
  constexpr int E = 16 / sizeof(T);  // elements per 16-byte chunk
  constexpr int CH = D / E;          // chunks per token-head row
  __shared__ T tile[kBlock][D + E];
  __shared__ int32_t slot_sh[kBlock];
  const int t0 = blockIdx.x * kBlock, h = blockIdx.y, tid = threadIdx.x;
  const int64_t limit = int64_t(num_blocks) * kBlock;
  if (tid < kBlock) {
    const int tok = t0 + tid;
    const int s = tok < n_tokens ? slots[tok] : -1;
    slot_sh[tid] = (s >= 0 && s < limit) ? s : -1;
  }
  __syncthreads();
  for (int c = tid; c < kBlock * CH; c += 256) {
    const int tt = c / CH, part = c % CH;
    const int tok = t0 + tt;
    const int s = slot_sh[tt];
    const int64_t src = ((int64_t)tok * hkv + h) * D + part * E;
    u32x4 kx = zero16(), vx = zero16();
    if (s >= 0) {
      // the new tokens' rows are read once: non-temporal loads keep them out of
      // the caches the attention call that follows re-reads
      kx = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(k_new + src));
      vx = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(v_new + src));
      const int blk = s / kBlock, off = s % kBlock;
      st16(kc + ((int64_t)blk * hkv + h) * kBlock * D + key_elem(off, part * E), kx);
    }
    st16(&tile[tt][part * E], vx);
  }
  __syncthreads();
  // The tile's tokens fill one cache block in order (a sequence's run of
  // new tokens starting on a block boundary): each thread writes eight
  // tokens of one dimension of V^T as one 16-byte store.
  const int s0 = slot_sh[0];
  bool in_order = s0 >= 0 && s0 % kBlock == 0;
#pragma unroll
  for (int tt = 1; tt < kBlock; ++tt) in_order = in_order && slot_sh[tt] == s0 + tt;
  if (in_order) {
    T* vb = vc + ((int64_t)(s0 / kBlock) * hkv + h) * D * kBlock;
    for (int c = tid; c < D * (kBlock / E); c += 256) {
      const int d = c / (kBlock / E), t8 = (c % (kBlock / E)) * E;
      T w[E];
#pragma unroll
      for (int i = 0; i < E; ++i) w[i] = tile[t8 + i][d];
      st16(vb + d * kBlock + t8, __builtin_bit_cast(u32x4, w));
    }
    return;
  }
  for (int e = tid; e < kBlock * D; e += 256) {
    const int tt = e % kBlock, d = e / kBlock;
    const int s = slot_sh[tt];
    if (s < 0) continue;
    const int blk = s / kBlock, off = s % kBlock;
    vc[(((int64_t)blk * hkv + h) * D + d) * kBlock + off] = tile[tt][d];
  }
}

template <typename T>
int launch_t(const void* kn, const void* vn, const int32_t* slots, int32_t n, void* kc, void* vc,
             int32_t nb, int32_t hkv, int32_t d, hipStream_t stream) {
  dim3 grid((n + kBlock - 1) / kBlock, hkv);
  if (d == 128)
    hipLaunchKernelGGL((kv_append_kernel<T, 128>), grid, dim3(256), 0, stream,
                       static_cast<const T*>(kn), static_cast<const T*>(vn), slots, n,
                       static_cast<T*>(kc), static_cast<T*>(vc), nb, hkv);
  else
    hipLaunchKernelGGL((kv_append_kernel<T, 64>), grid, dim3(256), 0, stream,
                       static_cast<const T*>(kn), static_cast<const T*>(vn), slots, n,
                       static_cast<T*>(kc), static_cast<T*>(vc), nb, hkv);
  return static_cast<int>(hipGetLastError());
}

}  // namespace

int launch_kv_append(const void* kn, const void* vn, const int32_t* slots, int32_t n, void* kc,
                     void* vc, int32_t nb, int32_t hkv, int32_t d, int32_t dtype,
                     hipStream_t stream) {
  if (n == 0) return 0;
  if (dtype == 1) return launch_t<__bf16>(kn, vn, slots, n, kc, vc, nb, hkv, d, stream);
  return launch_t<float>(kn, vn, slots, n, kc, vc, nb, hkv, d, stream);
}

}  // namespace dev
}  // namespace pa
