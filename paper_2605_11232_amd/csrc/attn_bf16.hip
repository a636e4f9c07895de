// bf16 paged attention over a prefix-shared KV cache on CDNA4 MFMA.
//
// What is computed (paper: Section 2, PagedAttention's block table and
// Automatic Prefix Caching; Section 3, cached shared prefixes give the result
// of recomputing them): for each query row, softmax(scale * q K^T) V over the
// keys 0..a of its sequence, where a is the query's logical position, keys
// and values gathered block by block through the block table.
//
// Item kinds of one launch (see plan.cpp):
//  * tile items, one workgroup of 4 wavefronts x 32 rows: 64-key steps of K
//    and V^T are copied from the paged cache straight into LDS (two stages)
//    and shared by the four wavefronts; S^T = K Q^T and O^T += V^T P^T run on
//    32x32x16 MFMA.  Computing the transposed score tile puts one query row
//    in each lane, so the online-softmax row max needs a single cross-lane
//    exchange, and the probabilities are already laid out as the B operand
//    of the PV product (no LDS round trip for P).
//  * shared-prefix items: the tile path over gathered rows of sequences whose
//    leading blocks coincide (cascade); partial results are merged.
//  * row items, one wavefront each: up to 32 rows (decode's G rows, or a
//    verification sequence's n_q * G rows cut in pieces) as one or two
//    16-column tiles of 16x16x32 MFMA, with K and V^T streamed straight from
//    HBM into registers over a split of the key range.
//
// The key order inside a tile is permuted so that each lane's eight PV
// k-elements are eight consecutive keys: then V^T operands are single 16-byte
// reads of the cache's [head_dim][block] value layout.
//
// Scores are scaled by scale * log2(e) and exponentiated with exp2; the
// natural-log LSE is recovered as ln2 * (m + log2 l).
#include <hip/hip_ext.h>

#include "device_common.h"
#include "plan_format.h"

namespace pa {
namespace dev {
namespace {

struct AttnArgs {
  const __bf16* q;
  const __bf16* kc;
  const __bf16* vc;
  const int32_t* bt;
  const int32_t* seq_lens;
  const int32_t* cu_q;
  const int32_t* plan;
  __bf16* out;
  float* lse;
  float* ws_o;
  float* ws_lse;
  int32_t max_blocks;
  int32_t num_blocks;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  float scale_log2;
};

// Row r of a tile's K buffer holds key perm32(r): bits 2 and 3 swapped.
__device__ __forceinline__ int perm32(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}

// Tile items walk the keys in steps of kTileSub 32-key sub-tiles (2 kTileSub
// cache blocks).  Smaller steps halve the LDS and registers a workgroup holds,
// so more workgroups share a CU.
#ifndef PA_TILE_SUB
#define PA_TILE_SUB 2
#endif
constexpr int kTileSub = PA_TILE_SUB;
static_assert(kTileSub == 1 || kTileSub == 2, "32- or 64-key tile steps");
constexpr int kTileWavesPerEu = kTileSub == 1 ? 3 : 2;

// LDS of a tile item: K and V^T of two steps, each step held as the cache's
// own 2 NSUB blocks (the grouped key layout [D/32][16 slots][32] for K,
// [D][16 keys] for V^T).  Blocks are copied straight from global memory into
// LDS (no register staging), each 64-unit (1 KB) piece of LDS from one
// contiguous 1 KB of the cache; the 16-byte units are XOR-swizzled within a
// piece so that the MFMA operand reads of 16 consecutive lanes fall in
// distinct banks:
//  K:   block b, 32-dim group c, slot position s, 8-dim unit p
//         -> unit (b D/32 + c) 64 + 4 s + (p ^ (s / 4 % 4))
//  V^T: dim row d, half h (8 keys)         -> unit 2 d + (h ^ vswz(d))
// Slot position s of a block holds offset s with bits 2 and 3 swapped, so
// row r of a step's 32-key tile (position r % 16 of its block) holds key
// 32 * (r / 32) + perm32(r % 32).
template <int D, int NSUB>
struct TileSmem {
  static constexpr int BLK = kBlock * D;  // bf16 per block of K or V^T
  __bf16 k[2][2 * NSUB * BLK];
  __bf16 v[2][2 * NSUB * BLK];
};

__device__ __forceinline__ int vswz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

// Cache-policy bits of a buffer load on gfx950: non-temporal.
constexpr int kCachePolicyNonTemporal = 2;

// s_waitcnt vmcnt(0): every global load of this wavefront, including the
// copies into LDS, has completed.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Asynchronous copy of 16 bytes per lane into LDS: lane l reads bytes
// [off, off + 16) of the wave-uniform block `base` (a buffer resource in
// scalar registers, so the per-copy address work is scalar) and writes them
// to bytes [16 l, 16 l + 16) after `lds` (wave-uniform).  Offsets at or past
// `bytes` read zeros instead of faulting.
// STREAM: the non-temporal cache policy (data read once: the lines are not
// kept in L2 at the expense of data other items re-read).
template <bool STREAM = false>
__device__ __forceinline__ void copy16_to_lds(const void* base, int bytes, uint32_t off, __bf16* lds) {
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0,
                                           STREAM ? kCachePolicyNonTemporal : 0);
}

// Sum of the eight bf16 values of a vector added to acc (v_dot2 with ones).
__device__ __forceinline__ float add_bf16x8(bf16x8 v, float acc) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    acc = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{v[2 * i], v[2 * i + 1]}, one, acc, false);
  return acc;
}

#ifndef PA_LDS_PREFETCH
#define PA_LDS_PREFETCH 3
#endif
// N MFMAs whose A operands are 16-byte LDS reads (addr(i) gives the address
// of MFMA i), with PF reads in flight ahead of the MFMA that uses them: LDS
// latency is hidden behind the MFMAs instead of being paid before each one.
// The scheduling-group barriers keep the read-ahead order in the code.
template <int N, int PF, class AddrF, class MfmaF>
__device__ __forceinline__ void lds_mfma_pipeline(AddrF addr, MfmaF mfma) {
  static_assert(PF >= 1 && PF <= N, "read-ahead depth");
  u32x4 x[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i) x[i] = ld16(addr(i));
  __builtin_amdgcn_sched_group_barrier(0x100, PF, 0);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const u32x4 a = x[i % PF];
    if (i + PF < N) {
      x[i % PF] = ld16(addr(i + PF));
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    mfma(i, a);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
}

// max of a value over the two lane halves (lane l and l ^ 32)
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Tile item (SHARED = false): 128 rows of one sequence, causal.  Shared-prefix
// item (SHARED = true): 128 gathered rows of a cascade group's members over
// keys every one of them sees; results go to the members' partial rows.
//
// Software pipeline over steps, one workgroup barrier per step: while the
// softmax of step t runs on the VALU, the score MFMAs of step t + 1 run on the
// matrix cores, and the PV MFMAs of step t overlap the row maxima of step
// t + 1.  K of step t + 2 and V^T of step t + 1 are copied into the LDS
// buffers freed by steps t and t - 1 during step t.
template <int D, int NSUB, bool SHARED, bool FULL, bool STREAM = false>
__device__ __forceinline__ void tile_item(const int32_t* it, int g, int poff, const AttnArgs& a,
                                          TileSmem<D, NSUB>& sm) {
  constexpr int KT = 32 * NSUB;     // keys per step
  constexpr int NB = KT / kBlock;   // blocks per step
  constexpr int NI = NSUB * D / 64; // LDS copies per wavefront per step, for each of K and V^T
  constexpr int BLK = TileSmem<D, NSUB>::BLK;
  const int tid = threadIdx.x, lane = tid & 63, j = lane & 31, hh = lane >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;
  const int G = a.group;
  const int lr = w * 32 + j;
  const int row0 = it[I_ROW0], nrows = it[I_NROWS], kv0 = it[I_KV0];
  const bool valid = lr < nrows;
  int key_seq, kend, qs, qi, hq, apos, wg_amin, part;
  if constexpr (SHARED) {
    // gathered row -> member sequence and its own row
    const int rpm = it[S_RPM];
    const int rg = row0 + lr;
    const int mi = rg / rpm, rl = rg - mi * rpm;
    const int32_t* mem = a.plan + it[S_MEMBERS] + 2 * (valid ? mi : 0);
    const int seq = mem[0];
    qs = a.cu_q[seq];
    qi = rl / G;
    hq = g * G + (rl - qi * G);
    part = mem[1] + poff + rl;
    key_seq = it[S_BLOCK_SEQ];
    kend = it[S_KV1];
    apos = valid ? kend - 1 : -1;  // every shared key is visible
    wg_amin = kend - 1;            // only a partial last step is masked
  } else {
    const int r = it[I_SEQ];
    const int L = a.seq_lens[r];
    qs = a.cu_q[r];
    const int n = a.cu_q[r + 1] - qs;
    const int rho = row0 + lr;
    qi = rho / G;
    hq = g * G + (rho - qi * G);
    part = it[I_PART] < 0 ? -1 : it[I_PART] + poff + lr;
    key_seq = r;
    kend = min(it[I_KV1], L);
    apos = valid ? L - n + qi : -1;
    // Rows are ordered by query, so the item's first row has the smallest
    // position: steps entirely at or below it need no causal mask.
    wg_amin = L - n + row0 / G;
  }

  bf16x8 qf[D / 16];
  {
    const __bf16* qp = a.q + ((int64_t)(qs + qi) * a.hq + hq) * D + 8 * hh;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = as_bf16x8(valid ? ld16(qp + 16 * ks) : zero16());
  }
  f32x16 acc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[dt][e] = 0.f;
  // Running reference max m (raw scores) and this lane's partial row sum l
  // (the two lane halves hold disjoint keys of the same row; they are added
  // at the end).  p = exp2(c * s - mc) with c = scale * log2(e), mc = c * m.
  const float c = a.scale_log2;
  float m = kNegInf, mc = 0.f, l = 0.f;

  // Per-lane byte offsets of this wavefront's LDS copies inside a block: copy
  // i fills LDS units 64 * (4 i + w) + lane of the step buffer.
  uint32_t koff[NI], voff[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int U = 64 * (4 * i + w) + lane;
    // K: LDS piece 4 i + w is 32-dim group (4 i + w) % (D/32) of a block
    const int grp = (4 * i + w) % (D / kKeyGroup), pos = lane >> 2;
    const int unit = (lane & 3) ^ ((pos >> 2) & 3);
    koff[i] = (uint32_t)((grp * kBlock * kKeyGroup + pos * kKeyGroup + 8 * unit) * 2);
    const int u = U % (2 * D), d = u >> 1, h = (u & 1) ^ vswz(d);
    voff[i] = (uint32_t)((d * kBlock + 8 * h) * 2);
  }
  const int32_t* bt = a.bt + (int64_t)key_seq * a.max_blocks;
  const char* kbase = reinterpret_cast<const char*>(a.kc + (int64_t)g * kBlock * D);
  const char* vbase = reinterpret_cast<const char*>(a.vc + (int64_t)g * D * kBlock);
  const int64_t blk_bytes = (int64_t)a.hkv * kBlock * D * 2;  // one block, all kv-heads

  // Block ids of a step (wave-uniform), clamped into the cache when the
  // window of 64 table entries is fetched.  Blocks at or past kend read the
  // item's last block again, so every copy reads inside the cache; their keys
  // are masked and their values zeroed before use.  Steps advance NB blocks
  // from the window's first block, so a step's blocks never straddle two
  // windows: one window check per step.
  BlockWindow win;
  win.init(bt, kend > 0 ? (kend - 1) / kBlock : 0, a.num_blocks, kv0 / kBlock);
  // blk[b]: byte offset of the step's block b (all kv-heads per block), so
  // each block's address is computed once for its K and its V^T copies
  auto step_blocks = [&](int t0, int64_t (&blk)[NB]) {
    const int jb = t0 / kBlock;
    win.seek(jb);
#pragma unroll
    for (int b = 0; b < NB; ++b)
      blk[b] = (int64_t)((uint64_t)(uint32_t)win.at(jb + b) * (uint32_t)blk_bytes);  // ids >= 0
  };
  // Copy slot i of wavefront w lands in block (4 i + w) * 64 / (2 D) of the
  // step: block i for D = 128, block 2 i + w / 2 for D = 64.
  static_assert(NI >= 1, "at least one copy per wavefront");
  static_assert(D == 64 || D == 128, "head_dim 64 or 128");
  auto copy_block = [&](const int64_t (&blk)[NB], int i) {
    if constexpr (D == 128) return blk[i];
    else return blk[2 * i] + ((w >> 1) & 1) * (blk[2 * i + 1] - blk[2 * i]);  // no indexed array
  };
  // one (block, kv-head) of K or V^T: kBlock * D bf16 at the block's address
  constexpr int kHeadBytes = kBlock * D * 2;
  // STREAM items (keys no other item reads) copy with the non-temporal
  // policy, leaving L2 to the keys other items re-read (shared prefixes,
  // the other tiles of a long sequence).
  auto issue_k = [&](const int64_t (&blk)[NB], int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      copy16_to_lds<STREAM>(kbase + copy_block(blk, i), kHeadBytes, koff[i],
                            &sm.k[buf][512 * (4 * i + w)]);
  };
  auto issue_v = [&](const int64_t (&blk)[NB], int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      copy16_to_lds<STREAM>(vbase + copy_block(blk, i), kHeadBytes, voff[i],
                            &sm.v[buf][512 * (4 * i + w)]);
  };

  // LDS operand addresses: per lane, the byte offset of its K unit for each
  // k-step (row j of a 32-key tile; the swizzle depends on the k-step) and
  // of its V^T unit; buffers, 32-key tiles and 32-dim tiles add constants, so
  // with the buffer known at compile time every operand read is one
  // register plus an immediate offset.
  uint32_t kofs[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const int pos = j % kBlock;
    kofs[ks] = 16u * (((j / kBlock) * (D / kKeyGroup) + ks / 2) * 64 + 4 * pos +
                      ((2 * (ks % 2) + hh) ^ ((pos >> 2) & 3)));
  }
  const uint32_t vofs = 16u * (2 * j + (hh ^ vswz(j)));  // vswz(32 dt + j) == vswz(j)
  auto lds_at = [](const __bf16* base, uint32_t byte_off) {
    return reinterpret_cast<const __bf16*>(reinterpret_cast<const char*>(base) + byte_off);
  };

  // S^T[key][row] of a step for the wave's 32 rows: NSUB independent 32-key chains.
  auto scores = [&](auto buf_c, f32x16 (&s)[NSUB]) {
    constexpr int buf = decltype(buf_c)::value;
#pragma unroll
    for (int u = 0; u < NSUB; ++u)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[u][e] = 0.f;
    // MFMA i: k-step i / NSUB of 32-key chain i % NSUB
    lds_mfma_pipeline<D / 16 * NSUB, PA_LDS_PREFETCH>(
        [&](int i) { return lds_at(&sm.k[buf][32 * (i % NSUB) * D], kofs[i / NSUB]); },
        [&](int i, u32x4 k) { s[i % NSUB] = mfma32(as_bf16x8(k), qf[i / NSUB], s[i % NSUB]); });
  };
  auto mask = [&](int t0, f32x16 (&s)[NSUB]) {
#pragma unroll
    for (int u = 0; u < NSUB; ++u)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = t0 + 32 * u + perm32(8 * (e >> 2) + 4 * hh + (e & 3));
        s[u][e] = key <= apos ? s[u][e] : kNegInf;
      }
  };
  auto rowmax = [&](const f32x16 (&s)[NSUB]) {
    float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
    for (int u = 0; u < NSUB; ++u)
#pragma unroll
      for (int e = (u == 0 ? 2 : 0); e < 16; e += 2) mx = fmaxf(fmaxf(mx, s[u][e]), s[u][e + 1]);
    return max_halves(mx);
  };
  // Move the reference max only when a score exceeds it by more than 2^8
  // (probabilities stay <= 256, exact in float32 sums and bf16 operands);
  // decided for the whole wavefront so every lane skips the rescale together.
  auto rebase = [&](float mx) {
    if (__any(mx != kNegInf && (m == kNegInf || mx * c > mc + 8.f))) {
      const float mnew = fmaxf(m, mx);
      const float mcn = mnew == kNegInf ? 0.f : mnew * c;
      const float alpha = m == kNegInf ? 0.f : fast_exp2(mc - mcn);
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[dt][e] *= alpha;
      m = mnew;
      mc = mcn;
    }
  };
  // Probabilities of a step as bf16 B operands: p[u][kk] holds keys
  // 32 u + 16 kk + 8 hh + 0..7 (the perm32 order makes them consecutive).
  // The row sum adds the bf16 probabilities the PV product uses, two per
  // v_dot2, in two chains.
  auto probs = [&](const f32x16 (&s)[NSUB], bf16x8 (&p)[NSUB][2]) {
#pragma unroll
    for (int u = 0; u < NSUB; ++u)
#pragma unroll
      for (int e = 0; e < 16; ++e) p[u][e >> 3][e & 7] = (__bf16)fast_exp2(fmaf(s[u][e], c, -mc));
    float l0 = l, l1 = 0.f;
#pragma unroll
    for (int u = 0; u < NSUB; ++u) {
      l0 = add_bf16x8(p[u][0], l0);
      l1 = add_bf16x8(p[u][1], l1);
    }
    l = l0 + l1;
  };
  auto pv = [&](auto buf_c, const bf16x8 (&p)[NSUB][2]) {
    constexpr int buf = decltype(buf_c)::value;
    // MFMA i: dims 32 (i % DT) .. of keys 16 (i / DT) .. (16-key half i / DT)
    constexpr int DT = D / 32;
    lds_mfma_pipeline<2 * NSUB * DT, PA_LDS_PREFETCH>(
        [&](int i) { return lds_at(&sm.v[buf][(i / DT) * BLK + 512 * (i % DT)], vofs); },
        [&](int i, u32x4 v) {
          acc[i % DT] = mfma32(as_bf16x8(v), p[(i / DT) / 2][(i / DT) % 2], acc[i % DT]);
        });
  };
  // Values of keys at or past kend in the last step: zero (never-written cache
  // slots may hold anything, and 0 * NaN would reach the output).
  auto zero_tail = [&](int t0, int buf) {
    const int nz = t0 + KT - kend;
    for (int x = tid; x < D * nz; x += 256) {
      const int d = x % D, k = kend - t0 + x / D;
      const int b = k / kBlock, kk = k % kBlock;
      sm.v[buf][b * BLK + 8 * (2 * d + ((kk >> 3) ^ vswz(d))) + (kk & 7)] = (__bf16)0.f;
    }
  };

  const int ntiles = kend > kv0 ? (kend - kv0 + KT - 1) / KT : 0;
  // steps [0, n_plain) need no causal or tail mask for any row of the item
  const int n_plain = min(ntiles, max(0, (wg_amin + 1 - kv0) / KT));
  if (ntiles > 0) {
    // blk[t % 2]: byte offsets of step t's blocks, found two steps ahead
    // (for the K copy) and used again one step ahead (for the V^T copy)
    int64_t blk[2][NB] = {};
    step_blocks(kv0, blk[0]);
    issue_k(blk[0], 0);
    issue_v(blk[0], 0);
    if (ntiles > 1) {
      step_blocks(kv0 + KT, blk[1]);
      issue_k(blk[1], 1);
    }
    wait_vmem();
    __syncthreads();
    // Wavefronts without rows (items of fewer than kTileRows rows) only help
    // with the copies and pass the barriers.
    const bool active = FULL || w * 32 < nrows;
    f32x16 s[NSUB];
    using B0 = std::integral_constant<int, 0>;
    using B1 = std::integral_constant<int, 1>;
    if (active) {
      scores(B0{}, s);
      if (n_plain == 0) mask(kv0, s);
      rebase(rowmax(s));
    }
    __syncthreads();  // K buffer 0 is refilled next

    // One pipelined step: softmax + PV of step t, scores + max of step t + 1.
    // buf_c = t % 2, the LDS buffer pair of step t (a compile-time constant).
    auto step = [&](int t, auto mask_next, auto buf_c) {
      constexpr int buf = decltype(buf_c)::value;
      const int t0 = kv0 + KT * t;
      if (t + 2 < ntiles) {
        step_blocks(t0 + 2 * KT, blk[buf]);
        issue_k(blk[buf], buf);
      }
      issue_v(blk[1 - buf], 1 - buf);  // blocks of step t + 1, found one step earlier
      bf16x8 p[NSUB][2];
      f32x16 sn[NSUB];
      probs(s, p);
      // The matrix section runs at raised issue priority: of the two
      // wavefronts sharing a SIMD, the one issuing MFMAs goes first and the
      // other's softmax VALU work fills the remaining issue slots.
      __builtin_amdgcn_s_setprio(1);
      scores(std::integral_constant<int, 1 - buf>{}, sn);
      // keep the row-sum additions in this region, where they overlap the
      // score MFMAs, instead of letting them sink past the barrier
      asm volatile("" : "+v"(l));
      pv(buf_c, p);
      __builtin_amdgcn_s_setprio(0);
      if constexpr (decltype(mask_next)::value) mask(t0 + KT, sn);
      const float mx = rowmax(sn);
      wait_vmem();
      __syncthreads();
      rebase(mx);
#pragma unroll
      for (int u = 0; u < NSUB; ++u) s[u] = sn[u];
    };
    auto idle_step = [&](int t, auto buf_c) {
      constexpr int buf = decltype(buf_c)::value;
      const int t0 = kv0 + KT * t;
      if (t + 2 < ntiles) {
        step_blocks(t0 + 2 * KT, blk[buf]);
        issue_k(blk[buf], buf);
      }
      issue_v(blk[1 - buf], 1 - buf);
      wait_vmem();
      __syncthreads();
    };
    // steps [t, lim) with the given masking, two at a time so that each
    // step's buffer pair is a compile-time constant
    auto run = [&](int& t, int lim, auto mask_next) {
      if (t < lim && (t & 1)) step(t++, mask_next, B1{});
      for (; t + 1 < lim; t += 2) {
        step(t, mask_next, B0{});
        step(t + 1, mask_next, B1{});
      }
      if (t < lim) step(t++, mask_next, B0{});
    };
    int t = 0;
    if (active) {
      // step t masks the scores of step t + 1: unmasked while t + 1 < n_plain
      run(t, min(n_plain, ntiles) - 1, std::false_type{});
      run(t, ntiles - 1, std::true_type{});
    } else {
      for (; t + 2 < ntiles; t += 2) {
        idle_step(t, B0{});
        idle_step(t + 1, B1{});
      }
      if (t + 1 < ntiles) idle_step(t++, B0{});
    }
    // last step: softmax + PV only
    const int t0 = kv0 + KT * t;
    bf16x8 p[NSUB][2];
    if (active) probs(s, p);
    if (t0 + KT > kend) {
      zero_tail(t0, t & 1);
      __syncthreads();
    }
    if (active) {
      if (t & 1) pv(B1{}, p);
      else pv(B0{}, p);
    }
  }

  l += wave_xor(l, 32);
  if (!valid) return;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse_v = l > 0.f ? kLn2 * (mc + __log2f(l)) : kNegInf;
  if (part < 0) {
    __bf16* op = a.out + ((int64_t)(qs + qi) * a.hq + hq) * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * dt + 8 * q4 + 4 * hh;
        __bf16 o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (__bf16)(acc[dt][4 * q4 + e] * inv);
        *reinterpret_cast<u32x2*>(op + d) = __builtin_bit_cast(u32x2, o4);
      }
    if (a.lse && hh == 0) a.lse[(int64_t)(qs + qi) * a.hq + hq] = lse_v;
  } else {
    float* op = a.ws_o + (int64_t)part * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int d = 32 * dt + 8 * q4 + 4 * hh;
        f32x4 o4;
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = acc[dt][4 * q4 + e] * inv;
        *reinterpret_cast<f32x4*>(op + d) = o4;
      }
    if (hh == 0) a.ws_lse[part] = lse_v;
  }
}

// Row item: one wavefront, up to 16 * NC rows (NC 16-column MFMA tiles that
// share every K and V^T operand), keys [kv0, kv1).  Decode items hold a
// sequence's G rows (NC = 1); verification items hold up to 32 of its
// n_q * G rows (NC = 2), so the keys are streamed from memory once per 32
// rows.  Sequences with more rows use tile items.
template <int D, int NC>
__device__ __forceinline__ void row_item(const int32_t* it, int g, int poff, const AttnArgs& a) {
  constexpr int KS = D / 32;  // k-steps of the QK product (32 dims each)
  constexpr int DT = D / 16;  // 16-row tiles of O^T
  const int r = it[I_SEQ];
  if (r < 0) return;
  const int row0 = it[I_ROW0], nrows = it[I_NROWS];
  const int kv0 = it[I_KV0], part = it[I_PART] < 0 ? -1 : it[I_PART] + poff;
  const int lane = threadIdx.x & 63, j = lane & 15, g4 = lane >> 4;
  const int L = a.seq_lens[r];
  const int qs = a.cu_q[r], n = a.cu_q[r + 1] - qs;
  // at most kRowItemBlocks blocks per item (the planner's limit; the clamp
  // keeps every table read inside the item's span)
  const int kv1 = min(min(it[I_KV1], L), kv0 + kRowItemBlocks * kBlock);
  const int G = a.group;

  // column j of tile c is the item's row 16 c + j
  bool valid[NC];
  int qi[NC], hq[NC], apos[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    valid[c] = 16 * c + j < nrows;
    const int rho = row0 + 16 * c + j;
    qi[c] = rho / G;
    hq[c] = g * G + (rho - qi[c] * G);
    apos[c] = valid[c] ? L - n + qi[c] : -1;
  }
  const int amin = L - n + row0 / G;  // smallest position among the item's rows

  bf16x8 qf[NC][KS];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const __bf16* qp = a.q + ((int64_t)(qs + qi[c]) * a.hq + hq[c]) * D + 8 * g4;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[c][ks] = as_bf16x8(valid[c] ? ld16(qp + 32 * ks) : zero16());
  }
  f32x4 acc[NC][DT];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[c][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float cs = a.scale_log2;
  float m[NC], mc[NC], l[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) m[c] = kNegInf, mc[c] = 0.f, l[c] = 0.f;

  const int32_t* bt = a.bt + (int64_t)r * a.max_blocks;
  const int64_t blk_k = (int64_t)a.hkv * kBlock * D, head_k = (int64_t)g * kBlock * D;
  const int64_t blk_v = (int64_t)a.hkv * D * kBlock, head_v = (int64_t)g * D * kBlock;
  // K operand row j of score tile tt holds key 8 * (j / 4) + 4 * tt + j % 4,
  // so each lane's score elements are eight consecutive keys (8 g4 .. + 7).

  // One register set for K and one for V^T: the next step's K loads are
  // issued as soon as the score MFMAs have consumed K, and its V^T loads as
  // soon as the PV MFMAs have consumed V^T, so HBM reads overlap the softmax
  // and the MFMAs of the current step.  The loads are non-temporal (private
  // keys are read once).  All loads are in bounds (a missing second block
  // aliases the first).
  u32x4 kreg[2][KS], vreg[DT];
  int b0 = 0, b1 = 0;
  BlockSpan win;
  win.init(bt, a.max_blocks, kv0 / kBlock);
  auto blocks_of = [&](int t0) {
    const int jb = t0 / kBlock;
    b0 = clamp_block(win.get(jb), a.num_blocks);
    b1 = t0 + 16 < kv1 ? clamp_block(win.get(jb + 1), a.num_blocks) : b0;
  };
  // That key sits in block j / 8 at slot position 8 tt + j % 8 (the grouped
  // key layout): each load reads, per block, eight
  // consecutive 64-byte slot rows of one 32-dim group, 512 contiguous bytes.
  auto load_k = [&]() {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int blk = j < 8 ? b0 : b1;
      const __bf16* p = a.kc + blk * blk_k + head_k + (8 * tt + (j & 7)) * kKeyGroup + 8 * g4;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kreg[tt][ks] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + kBlock * kKeyGroup * ks));
    }
  };
  auto load_v = [&]() {
    const __bf16* p = a.vc + (g4 < 2 ? b0 : b1) * blk_v + head_v + j * kBlock + 8 * (g4 & 1);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vreg[dt] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + 16 * kBlock * dt));
  };

  if (kv0 < kv1) {
    blocks_of(kv0);
    load_k();
    load_v();
  }
  for (int t0 = kv0; t0 < kv1; t0 += 32) {
    const bool more = t0 + 32 < kv1;
    f32x4 s[NC][2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        f32x4 acc_s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc_s = mfma16(as_bf16x8(kreg[tt][ks]), qf[c][ks], acc_s);
        s[c][tt] = acc_s;
      }
    if (more) {
      blocks_of(t0 + 32);
      load_k();
    }
    // Lane (j, g4), element e of score tile tt holds key t0 + 8 g4 + 4 tt + e.
    const bool masked = t0 + 31 > amin || !more;  // wave-uniform
    if (masked) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int key = t0 + 8 * g4 + 4 * tt + e;
            s[c][tt][e] = (key <= apos[c] && key < kv1) ? s[c][tt][e] : kNegInf;
          }
      // zero values of keys at or past kv1 (slots that may never have been written)
      const int keep = min(max(kv1 - (t0 + 8 * g4), 0), 8);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) vreg[dt] = keep_bf16(vreg[dt], keep);
    }
    bf16x8 pb[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float mx = fmaxf(fmaxf(s[c][0][0], s[c][0][1]), fmaxf(s[c][0][2], s[c][0][3]));
      mx = fmaxf(mx, fmaxf(fmaxf(s[c][1][0], s[c][1][1]), fmaxf(s[c][1][2], s[c][1][3])));
      mx = fmaxf(mx, wave_xor(mx, 16));
      mx = fmaxf(mx, wave_xor(mx, 32));
      if (__any(mx != kNegInf && (m[c] == kNegInf || mx * cs > mc[c] + 8.f))) {
        const float mnew = fmaxf(m[c], mx);
        const float mcn = mnew == kNegInf ? 0.f : mnew * cs;
        const float alpha = m[c] == kNegInf ? 0.f : fast_exp2(mc[c] - mcn);
        l[c] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[c][dt] *= alpha;
        m[c] = mnew;
        mc[c] = mcn;
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p = fast_exp2(fmaf(s[c][tt][e], cs, -mc[c]));
          l[c] += p;
          pb[c][4 * tt + e] = (__bf16)p;
        }
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int c = 0; c < NC; ++c) acc[c][dt] = mfma16(as_bf16x8(vreg[dt]), pb[c], acc[c][dt]);
    if (more) load_v();
  }

#pragma unroll
  for (int c = 0; c < NC; ++c) {
    l[c] += wave_xor(l[c], 16);
    l[c] += wave_xor(l[c], 32);
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (!valid[c]) continue;
    const float inv = l[c] > 0.f ? 1.f / l[c] : 0.f;
    const float lse_v = l[c] > 0.f ? kLn2 * (mc[c] + __log2f(l[c])) : kNegInf;
    if (part < 0) {
      __bf16* op = a.out + ((int64_t)(qs + qi[c]) * a.hq + hq[c]) * D + 4 * g4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        __bf16 o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (__bf16)(acc[c][dt][e] * inv);
        *reinterpret_cast<u32x2*>(op + 16 * dt) = __builtin_bit_cast(u32x2, o4);
      }
      if (a.lse && g4 == 0) a.lse[(int64_t)(qs + qi[c]) * a.hq + hq[c]] = lse_v;
    } else {
      const int prow = part + 16 * c + j;
      float* op = a.ws_o + (int64_t)prow * D + 4 * g4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) *reinterpret_cast<f32x4*>(op + 16 * dt) = acc[c][dt] * inv;
      if (g4 == 0) a.ws_lse[prow] = lse_v;
    }
  }
}

// MIX bits: 1 = tile and shared items, 2 = row items of at most 16 rows,
// 4 = row items of up to 32 rows, 8 = wildcard workgroups (tail lists).
// Separate instantiations keep a pure prefill or pure decode launch from
// paying the other paths' registers and LDS, and a plan without tail lists
// from paying for the wildcard loop; a launch with only 16-row row items
// runs at three waves per SIMD.
template <int MIX>
constexpr int waves_per_eu() { return MIX == 2 ? 3 : kTileWavesPerEu; }

template <int D, int MIX>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(waves_per_eu<MIX>()))) void attn_bf16_kernel(AttnArgs a) {
  const int32_t* plan = a.plan;
  // this workgroup's kv-head and template (the dispatch list follows the
  // header, so its word loads together with the header words); template
  // indices run over the shared, tile and row templates in that order
  const int wd = plan[kHeaderWords + blockIdx.x];
  const int g = wd >> kDispatchHeadShift, ti = wd & kDispatchIndexMask;
  const int n_shared = plan[H_N_SHARED_TMPL];
  const int n_tile = n_shared + plan[H_N_TILE_TMPL];  // templates before the row templates
  const int poff = g * plan[H_HEAD_PARTIAL];  // the kv-head's partial rows
  if constexpr (MIX & 1) {
    __shared__ TileSmem<D, kTileSub> sm;
    if constexpr ((MIX & 8) != 0) {
      if (ti == kWildcard) {
        // Take tail items (full tiles) from this XCD queue's list, then from
        // the other queues' lists while any has items left.  Each list has its
        // own counter in the plan (device-scope atomics, one cache line each);
        // the last wildcard workgroup to finish resets them, so the plan serves
        // the next call on the stream as uploaded.
        __shared__ int claim_sh;
        uint32_t* ctr = reinterpret_cast<uint32_t*>(const_cast<int32_t*>(plan)) + plan[H_CTR_OFF];
        const int32_t* tab = plan + plan[H_TAIL_OFF];
        const int32_t* tiles = plan + plan[H_TILE_OFF] - n_shared * kItemWords;
        const int home = blockIdx.x % kXcdQueues;  // the XCD queue this workgroup runs in
        // next item of list q, or past its end (every thread calls this)
        auto claim = [&](int q) {
          if (threadIdx.x == 0)
            claim_sh = int(__hip_atomic_fetch_add(ctr + q * kCounterWords, 1u, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT));
          __syncthreads();  // also: every wavefront is done with the previous item's LDS
          const int c = __builtin_amdgcn_readfirstlane(claim_sh);
          __syncthreads();  // claim_sh is written again next round
          return c;
        };
        auto run = [&](int q, int c) {
          const int tw = plan[tab[q] + c];
          const int tg = tw >> kDispatchHeadShift;
          tile_item<D, kTileSub, false, true>(tiles + (tw & kDispatchIndexMask) * kItemWords, tg,
                                              tg * plan[H_HEAD_PARTIAL], a, sm);
        };
        for (;;) {
          const int c = claim(home);
          if (c >= tab[kXcdQueues + home]) break;
          run(home, c);
        }
        // Other lists: one round trip reads their counters (lanes of the first
        // wavefront, atomic reads at the same coherence point as the claims)
        // and picks the first, in queue order after this one, with items left.
        // Every claim advances a counter, so the loop ends; the bound is a
        // second guarantee.
        for (int round = 0; round <= plan[H_N_TAIL] + kXcdQueues; ++round) {
          if (threadIdx.x < 64) {
            const int l = threadIdx.x;
            const int q = home + 1 + l < kXcdQueues ? home + 1 + l : home + 1 + l - kXcdQueues;
            bool left = false;
            if (l < kXcdQueues - 1)
              left = int(__hip_atomic_fetch_add(ctr + q * kCounterWords, 0u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT)) < tab[kXcdQueues + q];
            const uint64_t m = __ballot(left);
            if (l == 0) {
              const int f = m ? __builtin_ctzll(m) : -1;
              claim_sh = f < 0 ? -1 : (home + 1 + f) % kXcdQueues;
            }
          }
          __syncthreads();
          const int q = __builtin_amdgcn_readfirstlane(claim_sh);
          __syncthreads();
          if (q < 0) break;
          const int c = claim(q);
          if (c < tab[kXcdQueues + q]) run(q, c);
        }
        uint32_t* done = ctr + kXcdQueues * kCounterWords;
        if (threadIdx.x == 0 &&
            __hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1 ==
                uint32_t(plan[H_N_WILD])) {
          // every other wildcard workgroup has made its last claims
          for (int q = 0; q <= kXcdQueues; ++q)
            __hip_atomic_exchange(ctr + q * kCounterWords, 0u, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
      }
    }
    if (ti < n_shared) {
      const int32_t* it = plan + plan[H_SHARED_OFF] + ti * kSharedWords;
      if (it[S_NROWS] > kTileRows - 32) tile_item<D, kTileSub, true, true>(it, g, poff, a, sm);
      else tile_item<D, kTileSub, true, false>(it, g, poff, a, sm);
      return;
    }
    if (ti < n_tile) {
      const int32_t* it = plan + plan[H_TILE_OFF] + (ti - n_shared) * kItemWords;
      // every wavefront has rows: the plain path; otherwise idle ones skip
      // compute, and a few-row sequence's private keys are streamed
      if (it[I_NROWS] > kTileRows - 32) tile_item<D, kTileSub, false, true>(it, g, poff, a, sm);
      else if (it[I_FLAGS] & kItemStream) tile_item<D, kTileSub, false, false, true>(it, g, poff, a, sm);
      else tile_item<D, kTileSub, false, false>(it, g, poff, a, sm);
      return;
    }
  }
  if constexpr ((MIX & 6) != 0) {
    if (ti >= n_tile) {
      // a quad of row templates, one per wavefront
      const int32_t* it =
          plan + plan[H_ROW_OFF] + (ti - n_tile + (threadIdx.x >> 6)) * kItemWords;
      if constexpr ((MIX & 4) != 0) {
        if (it[I_NROWS] > 16) {
          row_item<D, 2>(it, g, poff, a);
          return;
        }
      }
      row_item<D, 1>(it, g, poff, a);
    }
  }
}

// Combine split partial results by log-sum-exp: one workgroup per merge
// group of at most four rows, half a wavefront per row (32 lanes over the
// output dims, 16-byte partial loads).  The partial outputs of up to 16 parts
// are requested before the part LSEs are reduced, so a row costs about one
// memory round trip; parts are combined in split order (deterministic).
template <int D>
__global__ __launch_bounds__(kMergeRows * 32) void merge_kernel(AttnArgs a) {
  constexpr int VD = D / 32;  // output dims per lane
  constexpr int C = 16;       // parts whose loads are in flight together
  typedef float vecf __attribute__((ext_vector_type(VD)));
  // merge group blockIdx.x: template blockIdx.x % N_GROUP_TMPL of kv-head
  // blockIdx.x / N_GROUP_TMPL
  const int ntg = a.plan[H_N_GROUP_TMPL];
  const int g = blockIdx.x / ntg;
  const int32_t* gr = a.plan + a.plan[H_GROUP_OFF] + (blockIdx.x - g * ntg) * kGroupWords;
  const int lr = threadIdx.x >> 5, lane = threadIdx.x & 31;
  const int half = threadIdx.x & 32;  // first lane of this row's half wavefront
  const int nrows = gr[G_NROWS];
  const bool valid = lr < nrows;
  const int r = gr[G_SEQ], row0 = gr[G_ROW0];
  const int nsplit = gr[G_NSPLIT], stride = gr[G_STRIDE];
  // partial row of split 0 (rows past nrows repeat the group's last row, in
  // bounds, and store nothing)
  const int64_t prow = (int64_t)gr[G_PART] + (int64_t)g * a.plan[H_HEAD_PARTIAL] + min(lr, nrows - 1);
  auto part_o = [&](int s) {
    return reinterpret_cast<const vecf*>(a.ws_o + (prow + (int64_t)s * stride) * D) + lane;
  };
  auto part_lse = [&](int s) { return a.ws_lse[prow + (int64_t)s * stride]; };
  vecf x[C];
  auto load_batch = [&](int s0) {
#pragma unroll
    for (int u = 0; u < C; ++u)
      if (s0 + u < nsplit) x[u] = *part_o(s0 + u);
  };
  load_batch(0);
  // max and sum of exp over the part LSEs, 32 parts per round
  const float lse0 = lane < nsplit ? part_lse(lane) : kNegInf;
  float mx = lse0;
  for (int s = 32 + lane; s - lane < nsplit; s += 32) mx = fmaxf(mx, s < nsplit ? part_lse(s) : kNegInf);
#pragma unroll
  for (int o = 16; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  vecf o_acc = {};
  float lse_v = kNegInf;
  if (mx != kNegInf) {
    float sum = lse0 == kNegInf ? 0.f : exp2f((lse0 - mx) * kLog2e);
    for (int s = 32 + lane; s - lane < nsplit; s += 32)
      if (s < nsplit) sum += exp2f((part_lse(s) - mx) * kLog2e);
#pragma unroll
    for (int o = 16; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    lse_v = mx + kLn2 * __log2f(sum);
    // weight of part s0 + lane of the current round of 32, held by that lane
    float wl = exp2f((lse0 - lse_v) * kLog2e);
    for (int s0 = 0; s0 < nsplit; s0 += C) {
      if (s0 > 0) {
        load_batch(s0);
        if (s0 % 32 == 0) {
          const int s = s0 + lane;
          wl = s < nsplit ? exp2f((part_lse(s) - lse_v) * kLog2e) : 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < C; ++u)
        if (s0 + u < nsplit) o_acc += __shfl(wl, half | ((s0 + u) & 31), 64) * x[u];
    }
  }
  if (!valid) return;
  const int qs = a.cu_q[r];
  const int rho = row0 + lr;
  const int qi = rho / a.group;
  const int hq = g * a.group + (rho - qi * a.group);
  __bf16 ob[VD];
#pragma unroll
  for (int k = 0; k < VD; ++k) ob[k] = (__bf16)o_acc[k];
  __bf16* op = a.out + ((int64_t)(qs + qi) * a.hq + hq) * D + VD * lane;
  if constexpr (VD == 4) *reinterpret_cast<u32x2*>(op) = __builtin_bit_cast(u32x2, ob);
  else *reinterpret_cast<uint32_t*>(op) = __builtin_bit_cast(uint32_t, ob);
  if (a.lse && lane == 0) a.lse[(int64_t)(qs + qi) * a.hq + hq] = lse_v;
}

}  // namespace

int launch_attn_bf16(const void* q, const void* kc, const void* vc, int32_t num_blocks,
                     const int32_t* bt, int32_t max_blocks, const int32_t* seq_lens,
                     const int32_t* cu_q, int32_t hq, int32_t hkv, int32_t d, float scale,
                     const int32_t* plan, int32_t grid, int32_t n_tile, int32_t n_groups,
                     bool wide_rows, bool tail, int64_t partial_rows, void* ws, void* out,
                     float* lse, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  AttnArgs a;
  a.q = static_cast<const __bf16*>(q);
  a.kc = static_cast<const __bf16*>(kc);
  a.vc = static_cast<const __bf16*>(vc);
  a.bt = bt;
  a.seq_lens = seq_lens;
  a.cu_q = cu_q;
  a.plan = plan;
  a.out = static_cast<__bf16*>(out);
  a.lse = lse;
  a.ws_o = static_cast<float*>(ws);
  a.ws_lse = a.ws_o ? a.ws_o + partial_rows * d : nullptr;
  a.max_blocks = max_blocks;
  a.num_blocks = num_blocks;
  a.hq = hq;
  a.hkv = hkv;
  a.group = hq / hkv;
  a.scale_log2 = scale * kLog2e;
  if (grid > 0) {
    // tiles and rows together: the tile path's register budget holds the
    // wide row path too
    const bool rows = grid > n_tile;
    const int mix = (n_tile == 0 ? (wide_rows ? 6 : 2) : (rows ? 7 : 1)) | (tail ? 8 : 0);
    // the caller's timing events ride on the dispatches (start on the first
    // kernel, stop on the last): no event packets between the kernels
    hipEvent_t stop_here = n_groups > 0 ? nullptr : ev_stop;
#define PA_LAUNCH(DD, MM)                                                                     \
  hipExtLaunchKernelGGL((attn_bf16_kernel<DD, MM>), dim3(grid), dim3(256), 0, stream, ev_start, \
                        stop_here, 0, a)
#define PA_LAUNCH_D(DD)                      \
  switch (mix) {                             \
    case 1: PA_LAUNCH(DD, 1); break;         \
    case 2: PA_LAUNCH(DD, 2); break;         \
    case 6: PA_LAUNCH(DD, 6); break;         \
    case 9: PA_LAUNCH(DD, 9); break;         \
    case 15: PA_LAUNCH(DD, 15); break;       \
    default: PA_LAUNCH(DD, 7); break;        \
  }
    if (d == 128) {
      PA_LAUNCH_D(128);
    } else {
      PA_LAUNCH_D(64);
    }
#undef PA_LAUNCH_D
#undef PA_LAUNCH
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return static_cast<int>(e);
  }
  if (n_groups > 0) {
    hipEvent_t start_here = grid > 0 ? nullptr : ev_start;
    if (d == 128)
      hipExtLaunchKernelGGL(merge_kernel<128>, dim3(n_groups), dim3(kMergeRows * 32), 0, stream,
                            start_here, ev_stop, 0, a);
    else
      hipExtLaunchKernelGGL(merge_kernel<64>, dim3(n_groups), dim3(kMergeRows * 32), 0, stream,
                            start_here, ev_stop, 0, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return static_cast<int>(e);
  }
  if (grid <= 0 && n_groups <= 0) {
    // nothing launched: the events still mark this point of the stream
    for (hipEvent_t ev : {ev_start, ev_stop}) {
      const hipError_t e = ev ? hipEventRecord(ev, stream) : hipSuccess;
      if (e != hipSuccess) return static_cast<int>(e);
    }
  }
  return 0;
}

}  // namespace dev
}  // namespace pa
