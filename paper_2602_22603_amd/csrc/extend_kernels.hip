// extend_kernels.hip - causal attention of a chunk of appended tokens over the
// paged, possibly compacted, KV cache, for gfx950 (CDNA4, wave64).
//
// Algorithm 1 grows the main thread's context by whole chunks (Phase 3: the
// turn's reasoning, then the tool output).  Each appended token attends to
// every cached key up to and including itself: the compacted prefix left by
// Phase 1's eviction and the chunk's earlier tokens.  Unlike decode this is a
// dense contraction (128 query rows share every K/V tile), so it runs on the
// matrix cores:
//
//   workgroup = 4 waves, 128 query rows = (128 / G tokens) x (G query heads
//               of one KV head); each wave owns 32 rows as two MFMA column
//               groups of 16.
//   K/V       = blocks of 64 keys (4 pages) staged in LDS, the next block's
//               global loads in flight while the current one is computed.
//   S^T       = K . Q^T      v_mfma_f32_16x16x32_bf16 (A = K rows from LDS,
//                            B = Q^T held in registers for the whole pass)
//   O^T      += V^T . P^T    v_mfma_f32_16x16x32_bf16 over 32 keys at once:
//               the k slots of lane group kg are keys 4kg..4kg+3 of two
//               consecutive 16-key tiles, which are exactly the S^T values
//               that lane already holds, so P never moves between lanes;
//               V^T is written to LDS in that slot order.  P is split into
//               bf16 hi + lo halves (two MFMAs) so the weights keep ~16 bits.
//   softmax   online, per query row, in log2 units (one v_exp_f32 per score);
//               row max across the four lane groups by permlane swaps.
//
// Work order: workgroup w takes KV head w % Hkv (consecutive workgroups land
// on different XCDs, so each XCD's L2 serves one head's K/V) and query block
// (n_qblocks - 1 - w / Hkv): the blocks that see the most keys start first.
#include <hip/hip_bf16.h>

#include "sq_kernels.hpp"

namespace sq {
namespace {

constexpr int BK = kExtKeys;
constexpr int kThreads = 256;
constexpr float kNegInf = -__builtin_huge_valf();

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

// bf16 round-to-nearest-even of two floats, packed low | high << 16.
__device__ inline uint32_t pack_bf16(float lo, float hi) {
  const __hip_bfloat162 v = __float22bfloat162_rn(make_float2(lo, hi));
  uint32_t u;
  __builtin_memcpy(&u, &v, sizeof(u));
  return u;
}

template <int D> struct ExtLayout {
  static constexpr int KP = D + 8;  // bf16 per LDS K row (16-byte pad: conflict-free A reads)
  static constexpr int VP = BK + 8; // bf16 per LDS V^T row
  static constexpr int NU = D / 32; // 16-byte K (and V) loads per thread per block
  static constexpr int E = 2 * D;   // 16-byte pieces per page and head
};

// Global -> registers: the K and V pieces of block blk this thread stages.
// Pages past the sequence's list read as zeros.
template <int D>
__device__ inline void ext_load(uint4 (&kr)[ExtLayout<D>::NU], uint4 (&vr)[ExtLayout<D>::NU],
                                const ExtendArgs &a, const uint16_t *kbase,
                                const uint16_t *vbase, int blk, int tid) {
  using Lt = ExtLayout<D>;
#pragma unroll
  for (int u = 0; u < Lt::NU; ++u) {
    const int c = u * kThreads + tid;
    const int p = c / Lt::E, w = c % Lt::E;
    const int pg = blk * (BK / kPage) + p;
    if (pg < a.n_pages) {
      const int64_t off = (int64_t)a.pt[pg] * a.page_stride + 8 * w;
      kr[u] = *reinterpret_cast<const uint4 *>(kbase + off);
      vr[u] = *reinterpret_cast<const uint4 *>(vbase + off);
    } else {
      kr[u] = make_uint4(0, 0, 0, 0);
      vr[u] = make_uint4(0, 0, 0, 0);
    }
  }
}

// Registers -> LDS.  K rows keep token order; V^T rows take the PV slot
// order (block key t = 32c + 16h + 4r + i  ->  slot 32c + 8r + 4h + i), and
// keys at or past L are zeroed so that 0 * v stays 0.
template <int D>
__device__ inline void ext_store(const uint4 (&kr)[ExtLayout<D>::NU], const uint4 (&vr)[ExtLayout<D>::NU],
                                 uint16_t *sk, uint16_t *sv, int blk, int tid, int L) {
  using Lt = ExtLayout<D>;
#pragma unroll
  for (int u = 0; u < Lt::NU; ++u) {
    const int c = u * kThreads + tid;
    const int p = c / Lt::E, w = c % Lt::E;
    const int tok = kPage * p + w / (D / 8);
    const int col = (w % (D / 8)) * 8;
    *reinterpret_cast<uint4 *>(sk + tok * Lt::KP + col) = kr[u];
    // V page is [D][16]: piece w holds channel w / 2, keys 8 (w % 2) .. +8
    const int d = w >> 1, h8 = w & 1;
    const int t0 = blk * BK + kPage * p + 8 * h8;
    uint4 x = vr[u];
    if (t0 + 8 > L) {
      uint32_t m[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        m[e] = (t0 + 2 * e < L ? 0xffffu : 0u) | (t0 + 2 * e + 1 < L ? 0xffff0000u : 0u);
      x.x &= m[0];
      x.y &= m[1];
      x.z &= m[2];
      x.w &= m[3];
    }
    const int s0 = 32 * (p >> 1) + 16 * h8 + 4 * (p & 1);
    *reinterpret_cast<uint2 *>(sv + d * Lt::VP + s0) = make_uint2(x.x, x.y);
    *reinterpret_cast<uint2 *>(sv + d * Lt::VP + s0 + 8) = make_uint2(x.z, x.w);
  }
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void k_extend(ExtendArgs a) {
  using Lt = ExtLayout<D>;
  constexpr int NKC = D / 32; // k chunks of S^T = K . Q^T
  constexpr int NDT = D / 16; // 16-channel tiles of O^T
  constexpr int TQ = kExtRows / G;
  __shared__ __attribute__((aligned(16))) uint16_t sk[BK * Lt::KP];
  __shared__ __attribute__((aligned(16))) uint16_t sv[D * Lt::VP];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 15, kg = lane >> 4;
  const int g = blockIdx.x % a.hkv;
  const int qb = a.n_qblocks - 1 - (int)(blockIdx.x / a.hkv);
  const int j0 = qb * TQ;
  const int base = a.L - a.n; // logical index of new token 0

  // this lane's two query columns (rows of the attention)
  bf16x8_t qf[2][NKC];
  int lim[2], jrow[2], hrow[2];
  bool live[2];
#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    const int c = 32 * wave + 16 * cg + n;
    jrow[cg] = j0 + c / G;
    hrow[cg] = g * G + c % G;
    live[cg] = jrow[cg] < a.n;
    lim[cg] = live[cg] ? base + jrow[cg] : a.L - 1;
    const uint16_t *qp = a.q + ((int64_t)jrow[cg] * a.hq + hrow[cg]) * D + 8 * kg;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const uint4 w = live[cg] ? *reinterpret_cast<const uint4 *>(qp + 32 * kc)
                               : make_uint4(0, 0, 0, 0);
      qf[cg][kc] = __builtin_bit_cast(bf16x8_t, w);
    }
  }
  const int kend = min(a.L, base + j0 + TQ); // keys this workgroup needs
  const int nblk = (kend + BK - 1) / BK;
  const int mask_from = base + j0;           // keys above this need the causal test

  f32x4_t acc[NDT][2];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) acc[dt][cg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {kNegInf, kNegInf}, l_run[2] = {0.f, 0.f};

  const uint16_t *kbase = a.k + (int64_t)g * a.head_stride;
  const uint16_t *vbase = a.v + (int64_t)g * a.head_stride;
  uint4 kr[Lt::NU], vr[Lt::NU];
  ext_load<D>(kr, vr, a, kbase, vbase, 0, tid);
  for (int b = 0; b < nblk; ++b) {
    if (b) __syncthreads(); // every wave is done reading the previous block
    ext_store<D>(kr, vr, sk, sv, b, tid, a.L);
    __syncthreads();
    if (b + 1 < nblk) ext_load<D>(kr, vr, a, kbase, vbase, b + 1, tid);

    f32x4_t st[4][2];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int cg = 0; cg < 2; ++cg) st[tt][cg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        const bf16x8_t ka = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4 *>(sk + (16 * tt + n) * Lt::KP + 32 * kc + 8 * kg));
#pragma unroll
        for (int cg = 0; cg < 2; ++cg)
          st[tt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[cg][kc], st[tt][cg], 0, 0, 0);
      }

    const bool need_mask = b * BK + BK - 1 > mask_from;
    uint4 phi[2][2], plo[2][2];
    float alpha[2];
#pragma unroll
    for (int cg = 0; cg < 2; ++cg) {
      float x[4][4];
      float mx = kNegInf;
#pragma unroll
      for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = b * BK + 16 * tt + 4 * kg + i;
          x[tt][i] = (need_mask && t > lim[cg]) ? kNegInf : st[tt][cg][i] * a.scale_log2;
          mx = fmaxf(mx, x[tt][i]);
        }
      mx = max_xrow16(mx);
      mx = max_xrow32(mx);
      const float m_new = fmaxf(m_run[cg], mx);
      const bool none = m_new == kNegInf;
      alpha[cg] = none ? 1.f : exp2_fast(m_run[cg] - m_new);
      float psum = 0.f;
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        uint32_t h[4], l[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int tt = 2 * c2 + (e >> 1);
          const float p0 = none ? 0.f : exp2_fast(x[tt][2 * (e & 1)] - m_new);
          const float p1 = none ? 0.f : exp2_fast(x[tt][2 * (e & 1) + 1] - m_new);
          h[e] = pack_bf16(p0, p1);
          l[e] = pack_bf16(p0 - bf_lo(h[e]), p1 - bf_hi(h[e]));
          psum += (bf_lo(h[e]) + bf_lo(l[e])) + (bf_hi(h[e]) + bf_hi(l[e]));
        }
        phi[cg][c2] = make_uint4(h[0], h[1], h[2], h[3]);
        plo[cg][c2] = make_uint4(l[0], l[1], l[2], l[3]);
      }
      l_run[cg] = l_run[cg] * alpha[cg] + psum;
      m_run[cg] = m_new;
    }
    if (__any(alpha[0] != 1.f || alpha[1] != 1.f)) {
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int cg = 0; cg < 2; ++cg) acc[dt][cg] *= alpha[cg];
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x8_t va = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4 *>(sv + (16 * dt + n) * Lt::VP + 32 * c2 + 8 * kg));
#pragma unroll
        for (int cg = 0; cg < 2; ++cg) {
          acc[dt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              va, __builtin_bit_cast(bf16x8_t, phi[cg][c2]), acc[dt][cg], 0, 0, 0);
          acc[dt][cg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              va, __builtin_bit_cast(bf16x8_t, plo[cg][c2]), acc[dt][cg], 0, 0, 0);
        }
      }
  }

#pragma unroll
  for (int cg = 0; cg < 2; ++cg) {
    float l = sum_xrow16(l_run[cg]);
    l = sum_xrow32(l);
    if (!live[cg]) continue;
    const float inv = 1.f / l;
    float *op = a.out + ((int64_t)jrow[cg] * a.hq + hrow[cg]) * D + 4 * kg;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
      *reinterpret_cast<float4 *>(op + 16 * dt) =
          make_float4(acc[dt][cg][0] * inv, acc[dt][cg][1] * inv, acc[dt][cg][2] * inv,
                      acc[dt][cg][3] * inv);
  }
}

template <int D> hipError_t extend_dispatch(int group, const ExtendArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)a.n_qblocks * (unsigned)a.hkv), block(kThreads);
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

hipError_t launch_extend(int d, int group, const ExtendArgs &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (d == 128) return extend_dispatch<128>(group, a, s);
  if (d == 64) return extend_dispatch<64>(group, a, s);
  return hipErrorInvalidValue;
}

} // namespace sq
