// extend_kernels.hip - causal attention of a chunk of appended tokens over the
// paged, possibly compacted, KV cache, for gfx950 (CDNA4, wave64).
//
// Algorithm 1 grows the main thread's context by whole chunks (Phase 3: the
// turn's reasoning, then the tool output).  Each appended token attends to
// every cached key up to and including itself: the compacted prefix left by
// Phase 1's eviction and the chunk's earlier tokens.  Unlike decode this is a
// dense contraction (256 query rows share every K/V tile), so it runs on the
// matrix cores:
//
//   workgroup = 8 waves (one workgroup per CU, two waves per SIMD), 256
//               query rows = (256 / G tokens) x (G query heads of one KV
//               head); each wave owns 32 rows as two MFMA column groups of
//               16.
//   K/V       = blocks of 64 keys (4 pages), copied global -> LDS by the
//               gfx950 direct-to-LDS buffer loads (16 bytes a lane) into
//               three buffers: blocks b + 1 and b + 2 are in flight while
//               block b is computed, and no registers hold staging data.  K
//               rows have their 16-byte chunks XOR-swizzled and V^T keeps
//               the pool's page layout, so that the MFMA operand reads below
//               are free of bank conflicts.
//   S^T       = K . Q^T      v_mfma_f32_16x16x32_bf16 (A = K rows from LDS,
//                            B = Q^T held in registers for the whole pass)
//   O^T      += V^T . P^T    v_mfma_f32_16x16x32_bf16 over 32 keys at once.
//               The A rows of the S^T tiles are chosen so that lane group kg
//               ends up holding the scores of keys 8kg .. 8kg+7 of each 32-key
//               chunk: exactly the k slots of its P^T operand and, in the
//               page-transposed V pool, one contiguous 16-byte piece of V^T.
//               P never moves between lanes.  P is split into bf16 hi + lo
//               halves (two MFMAs) so the weights keep ~16 bits.
//   softmax   online, per query row, in log2 units (one v_exp_f32 per score)
//               against a running reference that is raised only when the
//               weights of a half block could grow too large (see kBig); a
//               raise takes the half block's row maximum across the four
//               lane groups by permlane swaps.
//
// Work order: workgroup w takes KV head w % Hkv (consecutive workgroups land
// on different XCDs, so each XCD's L2 serves one head's K/V) and query block
// (n_qblocks - 1 - w / Hkv): the blocks that see the most keys start first.
#include <hip/hip_bf16.h>

#include "extend_args.hpp"
#include "fp8.hpp"

namespace sq {
namespace {

constexpr int BK = kExtKeys;
constexpr int kThreads = 64 * kExtWaves;
constexpr float kNegInf = -__builtin_huge_valf();
// Two waves per SIMD: the eight waves of the one workgroup a CU holds (up
// to 256 registers each).
constexpr int kExtWavesPerEu = 2;

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ inline float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ inline float bf_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

__device__ inline float max_xrow16(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float max_xrow32(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float sum_xrow16(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline float sum_xrow32(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));

// bf16 round-to-nearest-even of two floats, packed low | high << 16 (one
// v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2v_t));
}

template <int D> struct ExtLayout {
  static constexpr int CH = D / 8;             // 16-byte chunks per K row
  static constexpr int KROWS = 1024 / (2 * D); // K rows one wave-wide DMA writes
  static constexpr int K_ELEMS = BK * D;       // bf16 per K buffer
  static constexpr int V_ELEMS = D * BK;       // bf16 per V^T buffer
  static constexpr int NK = K_ELEMS * 2 / 1024 / kExtWaves; // K DMAs per wave per block
  static constexpr int NV = V_ELEMS * 2 / 1024 / kExtWaves; // V DMAs per wave per block
  static constexpr int PW = NK * KROWS;  // a wave's copies cover keys of page (wave * PW) / kPage
  static_assert(NK * kExtWaves * KROWS == BK && kPage % PW == 0, "a wave's copies stay in one page");
  static_assert(NV * 1024 == kPage * D * 2 * 4 / kExtWaves, "V^T copies split evenly");
};

// LDS layouts.  A 16-byte LDS read (ds_read_b128) is served half a wave at
// a time from 128 four-byte banks (measured on gfx950 with the
// bank-conflict counter), so it is conflict-free when the 32 chunks a
// half-wave reads are distinct modulo 32.
//   K: one row of D channels per key; an operand read has lane (n, kg) read
//      logical chunk 4 kc + kg of row tile_key(t, n) = 32a + 8(n >> 2) + 4h
//      + (n & 3), so chunks are XOR-swizzled within the row.  With 256-byte
//      rows the key (n & 3) + 4 (n >> 2) = n spreads the 8 rows of each
//      parity over all 16 slots; with 128-byte rows rows of equal n & 3
//      share a bank quarter, and 2 (n >> 2) separates them.
//   V^T: the block's four pages one after another, each as the pool holds
//      it (D rows of 16 keys, 32 bytes), so a page is copied as it lies.  A
//      P.V operand read has lane (n, kg) read keys 8 (4 c2 + kg) .. +7 of row
//      d = 16 dt + n: page 2 c2 + kg / 2, chunk 2 d + kg % 2 of it, which
//      makes 32 consecutive chunks per half-wave.
template <int D> __device__ inline int k_phys(int row, int c) {
  if constexpr (D == 128) return c ^ ((row & 3) + 4 * ((row >> 3) & 3));
  else return c ^ (2 * ((row >> 3) & 3));
}
// Element offset, in a V^T block buffer, of keys 8 j .. 8 j + 7 of row d.
template <int D> __device__ inline int v_off(int d, int j) {
  return (j >> 1) * (D * kPage) + d * kPage + 8 * (j & 1);
}

// The block key held by A row r of S^T tile t (0..3): tiles 2c and 2c + 1
// cover the 32-key chunk c, row 4 kg + i of tile 2c + h being key
// 32 c + 8 kg + 4 h + i.
__device__ inline int tile_key(int t, int r) {
  return 32 * (t >> 1) + 8 * (r >> 2) + 4 * (t & 1) + (r & 3);
}

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt immediate that waits until at most N vector memory operations
// are outstanding and leaves the other counters alone (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N> constexpr int kVmcntKeep = (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);

// A workgroup barrier for LDS written by ordinary stores: this wave's LDS
// stores complete, then the barrier.  __syncthreads() (and a fence on LDS
// alone) also waits for every vector memory operation in flight, the block
// copies into the other buffers included, since they too write LDS.  The
// memory clobber keeps the compiler from moving memory accesses across it.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Page ids of block blk (4 pages; ids past the sequence's list repeat its
// last page: every key there is at or past L, so its score is masked and its
// V zeroed before use).  The index is uniform, so these are scalar loads,
// issued a block ahead of their use.
// (Read through the constant address space: scalar loads, which the
// scalar-load counter tracks.  As vector loads, each wait for them would
// also wait for the block copies in flight, which count on the same
// in-order vector counter.)
typedef const int32_t __attribute__((address_space(4))) *ext_sptr_t;
__device__ inline void block_ids(int32_t (&ids)[4], const ExtendArgs &a, int blk) {
#pragma unroll
  for (int i = 0; i < 4; ++i) ids[i] = ((ext_sptr_t)a.pt)[min(blk * (BK / kPage) + i, a.n_pages - 1)];
}

// ids[q] for a q that may differ per lane, without branches.
__device__ inline int32_t pick4(const int32_t (&ids)[4], int q) {
  const int32_t lo = (q & 1) ? ids[1] : ids[0];
  const int32_t hi = (q & 1) ? ids[3] : ids[2];
  return (q & 2) ? hi : lo;
}

// A buffer resource over one page of a pool (the 16-byte loads below are
// relative to it).
__device__ inline __amdgpu_buffer_rsrc_t ext_page(const void *page, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(page), (short)0, bytes, 0x00020000);
}

// Global -> LDS (direct) for one block: each wave copies a part of one page
// of the block, K rows and V^T alike, so one page address per wave serves
// all of its copy instructions (formed by the scalar unit from the page id)
// and the lanes add offsets that do not change from block to block.
template <int D>
__device__ inline void ext_dma(uint16_t *sk, uint16_t *sv, const ExtendArgs &a,
                               const uint16_t *kbase, const uint16_t *vbase,
                               const int32_t (&ids)[4], int wave, int lane) {
  using Lt = ExtLayout<D>;
  constexpr int kPageBytes = kPage * D * 2;
  constexpr int IPP = kPageBytes / 1024; // copy instructions per page
  const int64_t off = (int64_t)pick4(ids, wave * Lt::PW / kPage) * a.page_stride;
  const __amdgpu_buffer_rsrc_t kr = ext_page(kbase + off, kPageBytes);
  const __amdgpu_buffer_rsrc_t vr = ext_page(vbase + off, kPageBytes);
#pragma unroll
  for (int u = 0; u < Lt::NK; ++u) {
    const int ins = wave * Lt::NK + u;
    const int row = ins * Lt::KROWS + lane / Lt::CH;
    const int c = k_phys<D>(row, lane % Lt::CH); // the swizzle is an involution
    __builtin_amdgcn_raw_ptr_buffer_load_lds(kr, (lds_void *)(sk + ins * 512), 16,
                                             ((row % kPage) * D + 8 * c) * 2, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < Lt::NV; ++u) {
    const int ins = wave * Lt::NV + u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(vr, (lds_void *)(sv + ins * 512), 16,
                                             ((ins % IPP) * 512 + lane * 8) * 2, 0, 0, 0);
  }
}

// An 8-bit store: the same block through registers.  ext_load8 loads the 8
// codes each lane's DMA would have copied as 8 bf16 values (half the bytes);
// ext_store8 converts them and writes the bf16 tile exactly where the DMA
// writes it, so the compute is unchanged.
template <int D>
__device__ inline void ext_load8(uint2 (&kr)[ExtLayout<D>::NK], uint2 (&vr)[ExtLayout<D>::NV],
                                 const ExtendArgs &a, const uint8_t *kbase, const uint8_t *vbase,
                                 const int32_t (&ids)[4], int wave, int lane) {
  using Lt = ExtLayout<D>;
#pragma unroll
  for (int u = 0; u < Lt::NK; ++u) {
    const int ins = wave * Lt::NK + u;
    const int row = ins * Lt::KROWS + lane / Lt::CH;
    const int c = k_phys<D>(row, lane % Lt::CH);
    const int p = (ins * Lt::KROWS) / kPage;
    kr[u] = *reinterpret_cast<const uint2 *>(kbase + (int64_t)pick4(ids, p) * a.page_stride +
                                             (row % kPage) * D + 8 * c);
  }
  constexpr int IPP = kPage * D * 2 / 1024; // bf16 copy instructions per page
#pragma unroll
  for (int u = 0; u < Lt::NV; ++u) {
    const int ins = wave * Lt::NV + u;
    vr[u] = *reinterpret_cast<const uint2 *>(vbase + (int64_t)pick4(ids, ins / IPP) * a.page_stride +
                                             (ins % IPP) * 512 + lane * 8);
  }
}
template <int D>
__device__ inline void ext_store8(uint16_t *sk, uint16_t *sv, const uint2 (&kr)[ExtLayout<D>::NK],
                                  const uint2 (&vr)[ExtLayout<D>::NV], int wave, int lane) {
  using Lt = ExtLayout<D>;
#pragma unroll
  for (int u = 0; u < Lt::NK; ++u) {
    const uint2 lo = e4m3x4_to_bf16(kr[u].x), hi = e4m3x4_to_bf16(kr[u].y);
    *reinterpret_cast<uint4 *>(sk + (wave * Lt::NK + u) * 512 + lane * 8) = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
#pragma unroll
  for (int u = 0; u < Lt::NV; ++u) {
    const uint2 lo = e4m3x4_to_bf16(vr[u].x), hi = e4m3x4_to_bf16(vr[u].y);
    *reinterpret_cast<uint4 *>(sv + (wave * Lt::NV + u) * 512 + lane * 8) = make_uint4(lo.x, lo.y, hi.x, hi.y);
  }
}

// Zero V^T entries of keys at or past L in the block's buffer (the last
// block only), so that 0 * v stays 0 whatever the pool holds there.
template <int D>
__device__ inline void ext_zero_tail(uint16_t *sv, int blk, int L, int tid) {
  for (int q = tid; q < D * 8; q += kThreads) {
    const int d = q >> 3, j = q & 7;
    const int k0 = blk * BK + 8 * j;
    if (k0 + 8 <= L) continue;
    uint4 *p = reinterpret_cast<uint4 *>(sv + v_off<D>(d, j));
    uint4 x = *p;
    uint32_t m[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      m[e] = (k0 + 2 * e < L ? 0xffffu : 0u) | (k0 + 2 * e + 1 < L ? 0xffff0000u : 0u);
    x.x &= m[0];
    x.y &= m[1];
    x.z &= m[2];
    x.w &= m[3];
    *p = x;
  }
}

// Softmax state of one lane: two query columns (rows of the attention).  m
// is the reference in log2 units: the weights of a half block (32 keys) are
// taken as 2^(s - m) against the m in hand, and only when some lane's sum of
// them reaches kBig (or the row has no reference yet) does the wave raise m
// to the half block's maximum, rescale O^T and l, and take the weights
// again.  A weight below 2^64 leaves fp32 room for l and acc over any key
// count, and out = acc / l does not depend on m.
constexpr float kBig = 0x1p64f;

// One 64-key block against this wave's 32 query columns.  need_mask: the
// block reaches past some column's last visible key (the chunk's diagonal,
// or the cache's end) or before some column's first one (a window), or holds
// slots a deferred eviction masked (lm: bit 4 tt + i = this lane's key
// tile_key(tt, 4 kg + i) is kept); only then is the per-key test made.
// after_scores() runs once the score MFMAs are issued: the caller's scalar
// loads go there, since while one is in flight (scalar loads return out of
// order on the counter they share with LDS reads) an MFMA could only wait
// for all 16 K reads at once instead of for its own.
template <int D, typename F>
__device__ __attribute__((always_inline)) inline void ext_block(const uint16_t *sk, const uint16_t *sv, int b, int n, int kg,
                                 float c, bool need_mask, const bf16x8_t (&qf)[2][D / 32],
                                 const int (&first)[2], const int (&lim)[2], uint32_t lm,
                                 f32x4_t (&acc)[D / 16][2], float (&m_run)[2], float (&l_run)[2],
                                 F &&after_scores) {
  constexpr int NKC = D / 32;
  constexpr int NDT = D / 16;
  f32x4_t st[4][2];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt)
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) st[tt][cg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // all the block's K fragments are read first (their LDS latency then
  // overlaps), k chunks outermost: the 8 accumulators of a block are 8
  // independent chains, so consecutive MFMAs never wait on each other's result
  bf16x8_t ka[NKC][4];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const int row = tile_key(tt, n);
      ka[kc][tt] = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const uint4 *>(sk + row * D + 8 * k_phys<D>(row, 4 * kc + kg)));
    }
  __builtin_amdgcn_sched_barrier(0); // (the compiler would move each read back next to its use)
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int cg = 0; cg < 2; ++cg)
        st[tt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[kc][tt], qf[cg][kc], st[tt][cg], 0, 0, 0);
  __builtin_amdgcn_sched_barrier(0);
  after_scores();
  if (need_mask) {
#pragma unroll
    for (int cg = 0; cg < 2; ++cg)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
        {
          const int key = b * BK + tile_key(tt, 4 * kg + i);
          if (key > lim[cg] || key < first[cg] || !((lm >> (4 * tt + i)) & 1)) st[tt][cg][i] = kNegInf;
        }
  }
  float nm[2];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) nm[cg] = m_run[cg] == kNegInf ? 0.f : -m_run[cg];
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    bf16x8_t phi[2], plo[2];
    float psum[2];
    auto weights = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int cg = 0; cg < 2; ++cg) {
        uint32_t h[4], l[4];
        psum[cg] = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int tt = 2 * c2 + (e >> 1);
          const float p0 = exp2_fast(fmaf(st[tt][cg][2 * (e & 1)], c, nm[cg]));
          const float p1 = exp2_fast(fmaf(st[tt][cg][2 * (e & 1) + 1], c, nm[cg]));
          h[e] = pack_bf16(p0, p1);
          l[e] = pack_bf16(p0 - bf_lo(h[e]), p1 - bf_hi(h[e]));
          psum[cg] += p0 + p1;
        }
        phi[cg] = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
        plo[cg] = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
      }
    };
    weights();
    const bool ok = m_run[0] != kNegInf && m_run[1] != kNegInf && psum[0] < kBig && psum[1] < kBig;
    if (!__all(ok)) { // (wave-uniform) raise the references to this half block's maxima
      float alpha[2];
#pragma unroll
      for (int cg = 0; cg < 2; ++cg) {
        float mx = kNegInf;
#pragma unroll
        for (int tt = 2 * c2; tt < 2 * c2 + 2; ++tt)
          mx = fmaxf(mx, fmaxf(fmaxf(st[tt][cg][0], st[tt][cg][1]), fmaxf(st[tt][cg][2], st[tt][cg][3])));
        mx = max_xrow16(mx);
        mx = max_xrow32(mx) * c; // scale > 0: the max commutes with it
        const float m_new = fmaxf(m_run[cg], mx);
        alpha[cg] = m_new == m_run[cg] ? 1.f : exp2_fast(m_run[cg] - m_new); // 0 from -inf
        m_run[cg] = m_new;
        nm[cg] = m_new == kNegInf ? 0.f : -m_new;
        l_run[cg] *= alpha[cg];
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int cg = 0; cg < 2; ++cg) acc[dt][cg] *= alpha[cg];
      weights();
    }
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) l_run[cg] += psum[cg];
    // all hi products, then all lo: the two MFMAs into one accumulator are
    // 2 * NDT instructions apart
    bf16x8_t va[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int d = 16 * dt + n;
      va[dt] = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const uint4 *>(sv + v_off<D>(d, 4 * c2 + kg)));
    }
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int cg = 0; cg < 2; ++cg)
        acc[dt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[dt], phi[cg], acc[dt][cg], 0, 0, 0);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int cg = 0; cg < 2; ++cg)
        acc[dt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[dt], plo[cg], acc[dt][cg], 0, 0, 0);
  }
}

template <int D, int G, bool KV8 = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(kExtWavesPerEu, kExtWavesPerEu))) void
k_extend(ExtendArgs a) {
  using Lt = ExtLayout<D>;
  constexpr int NKC = D / 32; // k chunks of S^T = K . Q^T
  constexpr int NDT = D / 16; // 16-channel tiles of O^T
  constexpr int TQ = kExtRows / G;
  // Three block buffers: block b is read from buffer b % 3 while the copies
  // of blocks b + 1 and b + 2 land in the other two.  They are separate LDS
  // objects and the block loop below is unrolled by three, so every LDS
  // read names its buffer at compile time: the compiler then knows that the
  // copies in flight cannot alias it and does not wait for them.
  __shared__ __attribute__((aligned(16))) uint16_t sk0[Lt::K_ELEMS], sk1[Lt::K_ELEMS], sk2[Lt::K_ELEMS];
  __shared__ __attribute__((aligned(16))) uint16_t sv0[Lt::V_ELEMS], sv1[Lt::V_ELEMS], sv2[Lt::V_ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6); // uniform: the DMA destination is M0
  const int n = lane & 15, kg = lane >> 4;
  const int g = blockIdx.x % a.hkv;
  const int rest = blockIdx.x / a.hkv;
  const int sp = rest % a.n_split; // key-range split
  const int qb = a.n_qblocks - 1 - rest / a.n_split;
  const int j0 = qb * TQ;
  const int base = a.L - a.n; // logical index of new token 0

  // this lane's two query columns (rows of the attention)
  bf16x8_t qf[2][NKC];
  int lim[2], first[2], jrow[2], hrow[2];
  bool live[2];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    const int col = 32 * wave + 16 * cg + n;
    jrow[cg] = j0 + col / G;
    hrow[cg] = g * G + col % G;
    live[cg] = jrow[cg] < a.n;
    lim[cg] = live[cg] ? base + jrow[cg] : a.L - 1;
    first[cg] = a.window > 0 ? lim[cg] - a.window + 1 : 0; // may be negative
    const uint16_t *qp = a.q + ((int64_t)jrow[cg] * a.hq + hrow[cg]) * D + 8 * kg;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const uint4 w = live[cg] ? *reinterpret_cast<const uint4 *>(qp + 32 * kc)
                               : make_uint4(0, 0, 0, 0);
      qf[cg][kc] = __builtin_bit_cast(bf16x8_t, w);
    }
  }
  const int kend = min(a.L, base + j0 + TQ); // keys this query block needs: [kbeg, kend)
  const int kbeg = a.window > 0 ? max(0, base + j0 - a.window + 1) : 0;
  const int b_lo = kbeg / BK + sp * a.split_blocks; // this workgroup's blocks [b_lo, b_hi)
  const int b_hi = min((kend + BK - 1) / BK, b_lo + a.split_blocks);
  const int mask_from = base + j0;           // keys above this need the causal test
  // keys below this are outside the window of the block's last token
  const int mask_below = a.window > 0 ? min(a.L - 1, base + j0 + TQ - 1) - a.window + 1 : 0;

  f32x4_t acc[NDT][2];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) acc[dt][cg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {kNegInf, kNegInf}, l_run[2] = {0.f, 0.f};

  const uint16_t *kbase = a.k + (int64_t)g * a.head_stride;
  const uint16_t *vbase = a.v + (int64_t)g * a.head_stride;
  const uint8_t *kbase8 = reinterpret_cast<const uint8_t *>(a.k) + (int64_t)g * a.head_stride;
  const uint8_t *vbase8 = reinterpret_cast<const uint8_t *>(a.v) + (int64_t)g * a.head_stride;
  uint2 kr[Lt::NK], vr[Lt::NV]; // an 8-bit store's next block, in flight
  int32_t ids[4];
  // Copies run two blocks ahead (one for an 8-bit store, whose next block
  // passes through registers): ids holds the page ids of the next block to
  // be fetched.  The copies of the two blocks past b_hi are issued too (of
  // the last page, block_ids clamps) into buffers that no block reads: with
  // a copy issued at the top of every block, the copies in flight at each
  // block's top are the same on every path, which the compiler can follow,
  // and it adds no wait of its own before the LDS reads.
  if (b_lo < b_hi) {
    block_ids(ids, a, b_lo);
    if constexpr (KV8) {
      ext_load8<D>(kr, vr, a, kbase8, vbase8, ids, wave, lane);
      ext_store8<D>(sk0, sv0, kr, vr, wave, lane);
    } else {
      ext_dma<D>(sk0, sv0, a, kbase, vbase, ids, wave, lane);
      // the query loads, issued before this copy, have landed (said here, on
      // the only way into the loop, so that the compiler knows it)
      __builtin_amdgcn_s_waitcnt(kVmcntKeep<Lt::NK + Lt::NV>);
      block_ids(ids, a, b_lo + 1);
      ext_dma<D>(sk1, sv1, a, kbase, vbase, ids, wave, lane);
    }
    block_ids(ids, a, KV8 ? b_lo + 1 : b_lo + 2);
    // block b from buffers c; buffers n1 and n2 are those of blocks b + 1 and
    // b + 2 (an 8-bit store uses only two buffers)
    auto block = [&](int b, uint16_t *ck, uint16_t *cv, uint16_t *n1k, uint16_t *n1v,
                     uint16_t *n2k, uint16_t *n2v) __attribute__((always_inline)) {
      // keep bits of this lane's 16 keys of the block (deferred evictions)
      uint32_t lm = 0xffffu;
      bool masked_here = false;
      if (a.masked) {
        const ext_sptr_t mr = (ext_sptr_t)a.mask_row;
        const int p0 = b * (BK / kPage), last = a.n_pages - 1;
        const uint32_t m0 = mr[min(p0, last)], m1 = mr[min(p0 + 1, last)];
        const uint32_t m2 = mr[min(p0 + 2, last)], m3 = mr[min(p0 + 3, last)];
        masked_here = (m0 & m1 & m2 & m3) != 0xffffu;
        if (masked_here) {
          // bit 4 tt + i is key tile_key(tt, 4 kg + i) = 32 (tt >> 1) + 8 kg
          // + 4 (tt & 1) + i: page 2 (tt >> 1) + (kg >> 1), slot 8 (kg & 1)
          // + 4 (tt & 1) + i, so tiles 0, 1 take 8 consecutive slots of page
          // kg >> 1 and tiles 2, 3 the same slots of page 2 + (kg >> 1)
          const int sh = 8 * (kg & 1);
          const uint32_t lo = (kg >> 1) ? m1 : m0, hi = (kg >> 1) ? m3 : m2;
          lm = ((lo >> sh) & 0xffu) | (((hi >> sh) & 0xffu) << 8);
        }
      }
      // block b has landed (every wave's copies; those of block b + 1, issued
      // later, may still be in flight) and every wave is done with block
      // b - 1, whose buffer the next copy overwrites
      __builtin_amdgcn_s_waitcnt(KV8 ? 0 : kVmcntKeep<Lt::NK + Lt::NV>);
      lds_barrier();
      if ((b + 1) * BK > a.L) {
        ext_zero_tail<D>(cv, b, a.L, tid);
        lds_barrier();
      }
      if constexpr (KV8) {
        if (b + 1 < b_hi) ext_load8<D>(kr, vr, a, kbase8, vbase8, ids, wave, lane); // stored after this block
      } else {
        ext_dma<D>(n2k, n2v, a, kbase, vbase, ids, wave, lane);
      }
      ext_block<D>(ck, cv, b, n, kg, a.scale_log2,
                   b * BK + BK - 1 > mask_from || b * BK < mask_below || masked_here, qf, first, lim,
                   lm, acc, m_run, l_run, [&]() __attribute__((always_inline)) {
                     if constexpr (KV8) {
                       if (b + 1 < b_hi) block_ids(ids, a, b + 2);
                     } else {
                       block_ids(ids, a, b + 3);
                     }
                   });
      if constexpr (KV8) { // a buffer every wave left by the top of this block
        if (b + 1 < b_hi) ext_store8<D>(n1k, n1v, kr, vr, wave, lane);
      }
    };
    if constexpr (KV8) {
      for (int b = b_lo; b < b_hi; b += 2) {
        block(b, sk0, sv0, sk1, sv1, sk0, sv0);
        if (b + 1 < b_hi) block(b + 1, sk1, sv1, sk0, sv0, sk1, sv1);
      }
    } else {
      // whole turns of the three buffers, then the rest: the loop's back
      // edge leaves every block of a turn behind it
      int b = b_lo;
      for (; b + 2 < b_hi; b += 3) {
        block(b, sk0, sv0, sk1, sv1, sk2, sv2);
        block(b + 1, sk1, sv1, sk2, sv2, sk0, sv0);
        block(b + 2, sk2, sv2, sk0, sv0, sk1, sv1);
      }
      if (b < b_hi) block(b, sk0, sv0, sk1, sv1, sk2, sv2);
      if (b + 1 < b_hi) block(b + 1, sk1, sv1, sk2, sv2, sk0, sv0);
      __builtin_amdgcn_s_waitcnt(0); // no copy lands in LDS after the workgroup ends
    }
  }

  if (a.n_split > 1) {
    // partial rows (a split may see no key of some rows: m = -inf, l = 0)
    const int64_t slot = ((int64_t)qb * a.hkv + g) * a.n_split + sp;
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) {
      float l = sum_xrow16(l_run[cg]);
      l = sum_xrow32(l);
      if (!live[cg]) continue;
      const int64_t row = slot * kExtRows + 32 * wave + 16 * cg + n;
      if (kg == 0) {
        a.part_m[row] = m_run[cg];
        a.part_l[row] = l;
      }
      float *pp = a.part_acc + row * D + 4 * kg;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
        *reinterpret_cast<float4 *>(pp + 16 * dt) =
            make_float4(acc[dt][cg][0], acc[dt][cg][1], acc[dt][cg][2], acc[dt][cg][3]);
    }
    return;
  }
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    float l = sum_xrow16(l_run[cg]);
    l = sum_xrow32(l);
    if (!live[cg]) continue;
    float sc = 1.f;
    if (a.sinks) { // one more term of the sum, no value: rescale both to the larger maximum
      const float sk_l2 = a.sinks[hrow[cg]] * a.sink_scale;
      const float big = fmaxf(m_run[cg], sk_l2);
      sc = exp2_fast(m_run[cg] - big);
      l = fmaf(l, sc, exp2_fast(sk_l2 - big));
    }
    const float inv = sc / l * a.out_scale;
    float *op = a.out + ((int64_t)jrow[cg] * a.hq + hrow[cg]) * D + 4 * kg;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
      *reinterpret_cast<float4 *>(op + 16 * dt) =
          make_float4(acc[dt][cg][0] * inv, acc[dt][cg][1] * inv, acc[dt][cg][2] * inv,
                      acc[dt][cg][3] * inv);
  }
}

// Merge of the split key range: one wave per (new token j, query head h),
// lanes over channels.  Its partials are row (j % TQ) * G + h % G of the
// n_split slots of (query block j / TQ, KV head h / G):
//   M = max m_s;  out = sum 2^(m_s - M) acc_s / sum 2^(m_s - M) l_s.
template <int D, int G>
__global__ __launch_bounds__(256) void k_extend_merge(ExtendArgs a) {
  constexpr int DPT = D / 64;
  constexpr int TQ = kExtRows / G;
  constexpr int U = 8;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); // (j, h) row
  if (r >= (int64_t)a.n * a.hq) return;
  const int j = (int)(r / a.hq), h = (int)(r % a.hq);
  const int g = h / G;
  const int64_t slot0 = ((int64_t)(j / TQ) * a.hkv + g) * a.n_split;
  const int col = (j % TQ) * G + h % G;
  const int S = a.n_split;
  float mine = kNegInf, lmine = 0.f;
  if (lane < S) {
    mine = a.part_m[(slot0 + lane) * kExtRows + col];
    lmine = a.part_l[(slot0 + lane) * kExtRows + col];
  }
  float big = mine;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) big = fmaxf(big, __shfl_xor(big, o));
  const float sink = a.sinks ? a.sinks[h] * a.sink_scale : kNegInf;
  big = fmaxf(big, sink);
  const float w = (lane < S && big != kNegInf) ? exp2_fast(mine - big) : 0.f;
  float den = w * lmine;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) den += __shfl_xor(den, o);
  if (a.sinks) den += exp2_fast(sink - big); // the sink's term, no value
  float num[DPT];
#pragma unroll
  for (int q = 0; q < DPT; ++q) num[q] = 0.f;
  for (int s0 = 0; s0 < S; s0 += U) {
    float x[U][DPT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sidx = min(s0 + u, S - 1);
      const float *p = a.part_acc + ((slot0 + sidx) * kExtRows + col) * D + lane * DPT;
#pragma unroll
      for (int q = 0; q < DPT; ++q) x[u][q] = p[q];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float wu = s0 + u < S ? __shfl(w, s0 + u) : 0.f;
#pragma unroll
      for (int q = 0; q < DPT; ++q) num[q] = fmaf(wu, x[u][q], num[q]);
    }
  }
  float *op = a.out + r * D + lane * DPT;
#pragma unroll
  for (int q = 0; q < DPT; ++q) op[q] = num[q] / den * a.out_scale;
}

template <int D> hipError_t extend_dispatch(int group, const ExtendArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)a.n_qblocks * (unsigned)a.hkv * (unsigned)a.n_split), block(kThreads);
  if (a.kv8) {
    switch (group) {
    case 1: hipLaunchKernelGGL((k_extend<D, 1, true>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_extend<D, 2, true>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_extend<D, 4, true>), grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_extend<D, 8, true>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (group) {
  case 1: hipLaunchKernelGGL((k_extend<D, 1>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_extend<D, 2>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_extend<D, 4>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_extend<D, 8>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

} // namespace

template <int D> hipError_t extend_merge_dispatch(int group, const ExtendArgs &a, hipStream_t s) {
  const int64_t rows = (int64_t)a.n * a.hq;
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_extend_merge<D, 1>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_extend_merge<D, 2>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_extend_merge<D, 4>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_extend_merge<D, 8>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_extend_merge(int d, int group, const ExtendArgs &a, hipStream_t s) {
  if (a.n <= 0 || a.n_split <= 1) return hipSuccess;
  if (d == 128) return extend_merge_dispatch<128>(group, a, s);
  if (d == 64) return extend_merge_dispatch<64>(group, a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_extend(int d, int group, const ExtendArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (d == 128) return extend_dispatch<128>(group, a, s);
  if (d == 64) return extend_dispatch<64>(group, a, s);
  return hipErrorInvalidValue;
}

} // namespace sq
