// decode_kernels.hip - decode-step attention over the paged, shared KV cache
// for gfx950 (CDNA4, wave64).
//
// Decode attention is the memory-bound step of long agentic contexts (§1;
// §3.4 "Compute and Memory Movement Cost").  One decode step of a batch of
// main-thread and auxiliary-thread queries (§3.1 "Parallel Execution") is
// split over work items (segment, KV head, chunk of pages), each producing
// an unnormalised partial (m, l, acc) per query row; a merge kernel combines
// the partials of every chunk a query attends to.
//
//   k_decode_valu  one query sequence per item: K and V page tiles staged in
//                  LDS, bf16 dot products on the VALU (v_dot2_f32_bf16), the
//                  online-softmax max and sum reduced with DPP and permlane
//                  swaps.
//   k_decode_mfma  up to four query sequences stacked as the 16 rows of an
//                  MFMA tile against the same pages - the prefix the main
//                  thread and its forked auxiliary thread share (§3.4 points
//                  to shared-prefix kernels for exactly this):
//                    S^T = K . Q^T  (v_mfma_f32_16x16x32_bf16, 16 tokens x 16 rows)
//                    O^T += V^T . P^T (v_mfma_f32_16x16x16_bf16, P split hi+lo)
//                  The S^T accumulator layout (lane = row + 16 * token group)
//                  is exactly the B operand P^T needs, so P never leaves its
//                  registers, and the page-transposed V pool is exactly the
//                  A operand V^T.
//   k_decode_merge M = max m_s; out = sum e^(m_s - M) acc_s / sum e^(m_s - M) l_s.
//
// Scores are kept in log2 units (scale * log2 e folded into one multiply) so
// every exponential is one v_exp_f32; m in the partials is in log2 units.
#include <hip/hip_bf16.h>

#include "sq_kernels.hpp"

namespace sq {
namespace {

constexpr int P = kPage;
constexpr float kNegInf = -__builtin_huge_valf();

typedef __bf16 bf16x2_t __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4_t __attribute__((__vector_size__(4 * sizeof(short))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ inline float bf_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ inline float bf_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

__device__ inline float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP moves within rows of 16 lanes.
template <int CTRL> __device__ inline float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kQuadXor1 = 0xB1; // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E; // quad_perm [2,3,0,1]
constexpr int kRowRor4 = 0x124;
constexpr int kRowRor8 = 0x128;

// The value of the partner 16 (resp. 32) lanes away, paired with our own:
// a permlane swap of x with itself leaves each lane holding {own, partner}.
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

struct ItemPos {
  Seg sg;
  int g;        // KV head
  int pbeg;     // first page (segment-local)
  int pend;     // one past the last page
  int npages;   // pages in the segment
};

__device__ inline ItemPos locate(const DecodeArgs &a, int item) {
  int lo = 0, hi = a.n_segs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].item0 <= item) lo = mid;
    else hi = mid - 1;
  }
  ItemPos ip;
  ip.sg = a.segs[lo];
  const int local = item - ip.sg.item0;
  ip.g = local / ip.sg.nchunk;
  const int c = local - ip.g * ip.sg.nchunk;
  ip.npages = (ip.sg.ntok + P - 1) / P;
  ip.pbeg = c * a.chunk_pages;
  ip.pend = min(ip.pbeg + a.chunk_pages, ip.npages);
  return ip;
}

// ===========================================================================
// VALU split-K kernel: one wave per item (one query sequence, one KV head).
//
// Lane roles per 16-token page:
//   scores  : lane = 4 * t + c  -> token t, channels {32 j + 8 c .. +8}
//             (G rows each), reduced over c inside the quad with DPP;
//             softmax of rows c, c+4, ... over t with DPP row rotations and
//             permlane swaps.
//   values  : lane = 4 * dg + R -> channels {dg * D/16 .. +D/16}, tokens
//             4R .. 4R+3; acc is partial over R and reduced at the end.
// LDS holds the page's K tile (row pitch 2D + 64 bytes) and V^T tile (groups
// of D/16 channels, 32 bytes per channel, 32 bytes of padding per group), the
// page's weights p[t][r] and the rescale factors alpha[r].
template <int D, int G>
__global__ __launch_bounds__(64) void k_decode_valu(DecodeArgs a) {
  constexpr int KPITCH = 2 * D + 64;
  constexpr int DPL = D / 16;
  constexpr int VGP = DPL * 32 + 32;
  constexpr int NLD = D / 32; // 16-byte loads per lane per tile
  constexpr int RPL = G >= 4 ? G / 4 : 1;
  __shared__ __attribute__((aligned(16))) unsigned char sK[P * KPITCH];
  __shared__ __attribute__((aligned(16))) unsigned char sV[16 * VGP];
  __shared__ __attribute__((aligned(16))) float sP[P * G];
  __shared__ __attribute__((aligned(16))) float sA[G];

  const int lane = threadIdx.x;
  const int item = a.item_begin + blockIdx.x;
  const ItemPos ip = locate(a, item);
  const int b = ip.sg.mem & 0xff;
  const int g = ip.g;
  const int32_t *pt = a.pt + (int64_t)ip.sg.row * a.max_pages + ip.sg.page0;

  const int t = lane >> 2, c = lane & 3; // score role
  const int R = lane & 3, dg = lane >> 2; // value role

  u32x4_t qr[G][NLD];
  {
    const uint16_t *qb = a.q + ((int64_t)b * a.hq + g * G) * D;
#pragma unroll
    for (int r = 0; r < G; ++r)
#pragma unroll
      for (int j = 0; j < NLD; ++j)
        qr[r][j] = *reinterpret_cast<const u32x4_t *>(qb + r * D + 32 * j + 8 * c);
  }

  float acc[G][DPL];
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[r][e] = 0.f;
  float m_run[RPL], l_run[RPL];
#pragma unroll
  for (int k = 0; k < RPL; ++k) {
    m_run[k] = kNegInf;
    l_run[k] = 0.f;
  }

  const uint16_t *kbase = a.k + (int64_t)g * P * D + lane * 8;
  const uint16_t *vbase = a.v + (int64_t)g * P * D + lane * 8;
  u32x4_t kreg[NLD], vreg[NLD];
  {
    const int64_t off = (int64_t)pt[ip.pbeg] * a.page_stride;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      kreg[i] = *reinterpret_cast<const u32x4_t *>(kbase + off + i * 512);
      vreg[i] = *reinterpret_cast<const u32x4_t *>(vbase + off + i * 512);
    }
  }

  for (int pg = ip.pbeg; pg < ip.pend; ++pg) {
    const int valid = (pg == ip.npages - 1) ? ip.sg.ntok - pg * P : P;
    // stage the page in LDS
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int e0 = i * 512 + lane * 8; // element offset inside the tile
      const int kt = e0 / D, kc = e0 % D;
      *reinterpret_cast<u32x4_t *>(sK + kt * KPITCH + kc * 2) = kreg[i];
      const int vd = e0 / P, vh = (e0 % P) / 8;
      *reinterpret_cast<u32x4_t *>(sV + (vd / DPL) * VGP + (vd % DPL) * 32 + vh * 16) = vreg[i];
    }
    __syncthreads();
    if (pg + 1 < ip.pend) { // prefetch the next page while this one is used
      const int64_t off = (int64_t)pt[pg + 1] * a.page_stride;
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        kreg[i] = *reinterpret_cast<const u32x4_t *>(kbase + off + i * 512);
        vreg[i] = *reinterpret_cast<const u32x4_t *>(vbase + off + i * 512);
      }
    }

    // scores: partial dot products over this lane's channels, then the quad
    float s[G];
#pragma unroll
    for (int r = 0; r < G; ++r) s[r] = 0.f;
#pragma unroll
    for (int j = 0; j < NLD; ++j) {
      const u32x4_t kv = *reinterpret_cast<const u32x4_t *>(sK + t * KPITCH + 64 * j + 16 * c);
#pragma unroll
      for (int r = 0; r < G; ++r) {
        s[r] = dot2(qr[r][j].x, kv.x, s[r]);
        s[r] = dot2(qr[r][j].y, kv.y, s[r]);
        s[r] = dot2(qr[r][j].z, kv.z, s[r]);
        s[r] = dot2(qr[r][j].w, kv.w, s[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < G; ++r) {
      s[r] += dpp<kQuadXor1>(s[r]);
      s[r] += dpp<kQuadXor2>(s[r]);
    }

    // online softmax for rows c + 4k (G >= 4) or c % G (G < 4), over t
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      const int row = G >= 4 ? c + 4 * k : c % G;
      float x = s[0];
#pragma unroll
      for (int r = 1; r < G; ++r) x = (row == r) ? s[r] : x;
      x = (t < valid) ? x * a.scale_log2 : kNegInf;
      float mx = x;
      mx = fmaxf(mx, dpp<kRowRor4>(mx));
      mx = fmaxf(mx, dpp<kRowRor8>(mx));
      mx = max_xrow16(mx);
      mx = max_xrow32(mx);
      const float m_new = fmaxf(m_run[k], mx);
      const bool none = m_new == kNegInf;
      const float alpha = none ? 1.f : exp2_fast(m_run[k] - m_new);
      const float pv = none ? 0.f : exp2_fast(x - m_new);
      l_run[k] = l_run[k] * alpha + pv;
      m_run[k] = m_new;
      if (G >= 4 || c < G) {
        sP[t * G + row] = pv;
        if (t == 0) sA[row] = alpha;
      }
    }
    __syncthreads();

    // values
    float al[G];
    bool rescale = false;
#pragma unroll
    for (int r = 0; r < G; ++r) {
      al[r] = sA[r];
      rescale |= al[r] != 1.f;
    }
    if (rescale) {
#pragma unroll
      for (int r = 0; r < G; ++r)
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[r][e] *= al[r];
    }
    float pw[4][G];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
      for (int r = 0; r < G; ++r) pw[tt][r] = sP[(4 * R + tt) * G + r];
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      const uint2 vv = *reinterpret_cast<const uint2 *>(sV + dg * VGP + e * 32 + 8 * R);
      float v0 = bf_lo(vv.x), v1 = bf_hi(vv.x), v2 = bf_lo(vv.y), v3 = bf_hi(vv.y);
      if (valid < P) { // values of absent tokens may be anything: keep 0 * v finite
        v0 = 4 * R + 0 < valid ? v0 : 0.f;
        v1 = 4 * R + 1 < valid ? v1 : 0.f;
        v2 = 4 * R + 2 < valid ? v2 : 0.f;
        v3 = 4 * R + 3 < valid ? v3 : 0.f;
      }
#pragma unroll
      for (int r = 0; r < G; ++r) {
        float y = acc[r][e];
        y = fmaf(pw[0][r], v0, y);
        y = fmaf(pw[1][r], v1, y);
        y = fmaf(pw[2][r], v2, y);
        y = fmaf(pw[3][r], v3, y);
        acc[r][e] = y;
      }
    }
    __syncthreads();
  }

  // sums over tokens and token quarters
  float l_tot[RPL];
#pragma unroll
  for (int k = 0; k < RPL; ++k) {
    float l = l_run[k];
    l += dpp<kRowRor4>(l);
    l += dpp<kRowRor8>(l);
    l = sum_xrow16(l);
    l = sum_xrow32(l);
    l_tot[k] = l;
  }
#pragma unroll
  for (int r = 0; r < G; ++r)
#pragma unroll
    for (int e = 0; e < DPL; ++e) {
      float y = acc[r][e];
      y += dpp<kQuadXor1>(y);
      y += dpp<kQuadXor2>(y);
      acc[r][e] = y;
    }

  const int64_t prow = (int64_t)item * kRows;
  if (t == 0 && (G >= 4 || c < G)) {
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
      const int row = G >= 4 ? c + 4 * k : c;
      a.part_m[prow + row] = m_run[k];
      a.part_l[prow + row] = l_tot[k];
    }
  }
  if (R == 0) {
#pragma unroll
    for (int r = 0; r < G; ++r) {
      float *dst = a.part_acc + (prow + r) * D + dg * DPL;
#pragma unroll
      for (int e = 0; e < DPL; e += 4)
        *reinterpret_cast<float4 *>(dst + e) =
            make_float4(acc[r][e], acc[r][e + 1], acc[r][e + 2], acc[r][e + 3]);
    }
  }
}

// ===========================================================================
// MFMA multi-query tile: one wave per item; up to 16 query rows (nmem
// sequences x G heads of one KV head) against the same pages.
// Lane l = n + 16 * kg (n = l & 15, kg = l >> 4):
//   QK A operand  K[token n][channels 8 kg + 32 s .. +8]       (16x16x32)
//   QK B operand  Q[row n][same channels]
//   S^T output    S[token 4 kg + i][row n], i < 4
//   PV A operand  V^T[channel n + 16 jd][tokens 4 kg .. +4]    (16x16x16)
//   PV B operand  P[row n][tokens 4 kg + i]  = the S^T registers after softmax
//   O^T output    O[row n][channel 16 jd + 4 kg + i]
// P is split into bf16 hi + lo parts (two MFMAs per block) so the weights
// keep ~16 bits; the running sum l uses the same hi + lo values.
template <int D, int G>
__global__ __launch_bounds__(64) void k_decode_mfma(DecodeArgs a) {
  constexpr int NS = D / 32;
  constexpr int NJ = D / 16;
  const int lane = threadIdx.x;
  const int n = lane & 15, kg = lane >> 4;
  const int item = a.item_begin + blockIdx.x;
  const ItemPos ip = locate(a, item);
  const int g = ip.g;
  const int nrows = ip.sg.nmem * G;
  const bool qvalid = n < nrows;
  const int jm = qvalid ? n / G : 0;
  const int bq = (ip.sg.mem >> (8 * jm)) & 0xff;
  const int32_t *pt = a.pt + (int64_t)ip.sg.row * a.max_pages + ip.sg.page0;

  bf16x8_t qb[NS];
  {
    const uint16_t *qp = a.q + ((int64_t)bq * a.hq + g * G + n % G) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      uint4 w = qvalid ? *reinterpret_cast<const uint4 *>(qp + 8 * kg + 32 * s)
                       : make_uint4(0, 0, 0, 0);
      qb[s] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  f32x4_t acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) acc[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;

  const uint16_t *kbase = a.k + (int64_t)g * P * D + n * D + 8 * kg;
  const uint16_t *vbase = a.v + (int64_t)g * P * D + n * P + 4 * kg;
  uint4 ka[NS];
  uint2 va[NJ];
  auto load_page = [&](int pg) {
    const int64_t off = (int64_t)pt[pg] * a.page_stride;
#pragma unroll
    for (int s = 0; s < NS; ++s) ka[s] = *reinterpret_cast<const uint4 *>(kbase + off + 32 * s);
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      va[j] = *reinterpret_cast<const uint2 *>(vbase + off + 16 * P * j);
  };
  load_page(ip.pbeg);

  for (int pg = ip.pbeg; pg < ip.pend; ++pg) {
    const int valid = (pg == ip.npages - 1) ? ip.sg.ntok - pg * P : P;
    uint4 kc[NS];
    uint2 vc[NJ];
#pragma unroll
    for (int s = 0; s < NS; ++s) kc[s] = ka[s];
#pragma unroll
    for (int j = 0; j < NJ; ++j) vc[j] = va[j];
    if (pg + 1 < ip.pend) load_page(pg + 1);

    f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
      st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kc[s]), qb[s],
                                                   st, 0, 0, 0);
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = (4 * kg + i < valid) ? st[i] * a.scale_log2 : kNegInf;
    float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mx = max_xrow16(mx);
    mx = max_xrow32(mx);
    const float m_new = fmaxf(m_run, mx);
    const bool none = m_new == kNegInf;
    const float alpha = none ? 1.f : exp2_fast(m_run - m_new);
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = none ? 0.f : exp2_fast(x[i] - m_new);
    const uint32_t h01 = pack_bf16(p[0], p[1]);
    const uint32_t h23 = pack_bf16(p[2], p[3]);
    const float r0 = p[0] - bf_lo(h01), r1 = p[1] - bf_hi(h01);
    const float r2 = p[2] - bf_lo(h23), r3 = p[3] - bf_hi(h23);
    const uint32_t l01 = pack_bf16(r0, r1);
    const uint32_t l23 = pack_bf16(r2, r3);
    const float psum = (bf_lo(h01) + bf_lo(l01)) + (bf_hi(h01) + bf_hi(l01)) +
                       (bf_lo(h23) + bf_lo(l23)) + (bf_hi(h23) + bf_hi(l23));
    l_run = l_run * alpha + psum;
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) acc[j] *= alpha;
    }
    if (valid < P) { // values of absent tokens may be anything: keep 0 * v finite
      const uint32_t m0 = (4 * kg + 0 < valid ? 0xffffu : 0u) | (4 * kg + 1 < valid ? 0xffff0000u : 0u);
      const uint32_t m1 = (4 * kg + 2 < valid ? 0xffffu : 0u) | (4 * kg + 3 < valid ? 0xffff0000u : 0u);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        vc[j].x &= m0;
        vc[j].y &= m1;
      }
    }
    const s16x4_t phi = __builtin_bit_cast(s16x4_t, make_uint2(h01, h23));
    const s16x4_t plo = __builtin_bit_cast(s16x4_t, make_uint2(l01, l23));
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const s16x4_t vA = __builtin_bit_cast(s16x4_t, vc[j]);
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vA, phi, acc[j], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vA, plo, acc[j], 0, 0, 0);
    }
  }

  float l_tot = sum_xrow16(l_run);
  l_tot = sum_xrow32(l_tot);
  if (qvalid) {
    const int64_t prow = (int64_t)item * kRows + n;
    if (kg == 0) {
      a.part_m[prow] = m_run;
      a.part_l[prow] = l_tot;
    }
    float *dst = a.part_acc + prow * D + 4 * kg;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      *reinterpret_cast<float4 *>(dst + 16 * j) = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
  }
}

// ===========================================================================
// Merge: one wave per (batch entry, query head).
template <int D>
__global__ __launch_bounds__(64) void k_decode_merge(MergeArgs a) {
  constexpr int DPT = D / 64;
  const int b = blockIdx.x / a.hq;
  const int h = blockIdx.x - b * a.hq;
  const int g = h / a.group;
  const int hr = h - g * a.group;
  const int ns = a.n_src[b];
  float big_m = kNegInf;
  for (int e = 0; e < ns; ++e) {
    const int nch = a.nchunk[b][e];
    const int row = a.member[b][e] * a.group + hr;
    const int64_t base = (int64_t)(a.item_base[b][e] + g * nch) * kRows + row;
    for (int c = 0; c < nch; ++c) big_m = fmaxf(big_m, a.part_m[base + (int64_t)c * kRows]);
  }
  float num[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) num[i] = 0.f;
  float den = 0.f;
  if (big_m != kNegInf) {
    for (int e = 0; e < ns; ++e) {
      const int nch = a.nchunk[b][e];
      const int row = a.member[b][e] * a.group + hr;
      const int64_t base = (int64_t)(a.item_base[b][e] + g * nch) * kRows + row;
      for (int c = 0; c < nch; ++c) {
        const int64_t idx = base + (int64_t)c * kRows;
        const float w = exp2_fast(a.part_m[idx] - big_m);
        den = fmaf(w, a.part_l[idx], den);
        const float *src = a.part_acc + idx * D + threadIdx.x * DPT;
#pragma unroll
        for (int i = 0; i < DPT; ++i) num[i] = fmaf(w, src[i], num[i]);
      }
    }
  }
  float *o = a.out + ((int64_t)b * a.hq + h) * D + threadIdx.x * DPT;
#pragma unroll
  for (int i = 0; i < DPT; ++i) o[i] = den > 0.f ? num[i] / den : 0.f;
}

template <int D>
hipError_t valu_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  const dim3 grid(a.n_items), block(64);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_decode_valu<D, 1>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_decode_valu<D, 2>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_valu<D, 4>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_valu<D, 8>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D>
hipError_t mfma_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  const dim3 grid(a.n_items), block(64);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_decode_mfma<D, 1>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_decode_mfma<D, 2>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_mfma<D, 4>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_mfma<D, 8>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

} // namespace

hipError_t launch_decode_valu(int d, int group, const DecodeArgs &a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  return d == 128 ? valu_dispatch<128>(group, a, s) : valu_dispatch<64>(group, a, s);
}

hipError_t launch_decode_mfma(int d, int group, const DecodeArgs &a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  return d == 128 ? mfma_dispatch<128>(group, a, s) : mfma_dispatch<64>(group, a, s);
}

hipError_t launch_decode_merge(int d, int batch, const MergeArgs &a, hipStream_t s) {
  const dim3 grid(batch * a.hq), block(64);
  if (d == 128)
    hipLaunchKernelGGL(k_decode_merge<128>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_decode_merge<64>, grid, block, 0, s, a);
  return hipGetLastError();
}

} // namespace sq
