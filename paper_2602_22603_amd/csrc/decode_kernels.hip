// decode_kernels.hip - decode-step attention over the paged, shared KV cache
// for gfx950 (CDNA4, wave64).
//
// Decode attention is the memory-bound step of long agentic contexts (§1;
// §3.4 "Compute and Memory Movement Cost").  One decode step of a batch of
// main-thread and auxiliary-thread queries (§3.1 "Parallel Execution") is
// split over workgroups that each take an equal share of the launch's
// (segment, KV head) page rows, writing an unnormalised partial (m, l, acc)
// per query row for every row piece they cover; a merge kernel combines the
// partials of every piece a query attends to.
//
//   k_decode_valu  one query sequence per item: K and V page tiles staged in
//                  LDS, bf16 dot products on the VALU (v_dot2_f32_bf16), the
//                  online-softmax max and sum reduced with DPP and permlane
//                  swaps.  In an 8-bit store each lane loads 8 codes and
//                  converts them to bf16 on the way into LDS.
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
// A decode step of the model appends one token per thread before it attends
// (Algorithm 1, Phase 3 grows the context token by token while decoding).
// k_step_valu / k_step_mfma / k_step_merge are the same kernels for a step
// whose plan lives in device memory (so a captured step replays for later
// steps); the step's merge adds each entry's new token as one more partial
// and stores it in the pools, which saves the append launch.
//
// Scores are kept in log2 units (scale * log2 e folded into one multiply) so
// every exponential is one v_exp_f32; m in the partials is in log2 units.
#include <hip/hip_bf16.h>

#include "decode_args.hpp"
#include "fp8.hpp"

#include <mutex>

namespace sq {
namespace {

constexpr int P = kPage;
constexpr float kNegInf = -__builtin_huge_valf();

typedef __bf16 bf16x2_t __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef short s16x4_t __attribute__((__vector_size__(4 * sizeof(short))));
typedef float f32x4_t __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// K/V page loads.  With NT (a page is read once per launch) they are
// non-temporal; when several sequences of one launch read the same pages the
// ordinary loads let L2 and the memory-side cache serve the repeats.
template <bool NT> __device__ inline u32x4_t ld_kv4(const uint16_t *p) {
  const u32x4_t *q = reinterpret_cast<const u32x4_t *>(p);
  if constexpr (NT) return __builtin_nontemporal_load(q);
  else return *q;
}
// Eight E4M3 codes (8 bytes) as eight bf16 values in one 16-byte register
// group, element order kept.
template <bool NT> __device__ inline u32x4_t ld_kv4_8(const uint8_t *p) {
  const u32x2_t *q = reinterpret_cast<const u32x2_t *>(p);
  u32x2_t x;
  if constexpr (NT) x = __builtin_nontemporal_load(q);
  else x = *q;
  const uint2 lo = e4m3x4_to_bf16(x.x), hi = e4m3x4_to_bf16(x.y);
  return u32x4_t{lo.x, lo.y, hi.x, hi.y};
}
template <bool NT> __device__ inline uint4 ld_stream(const uint16_t *p) {
  const u32x4_t x = ld_kv4<NT>(p);
  return make_uint4(x.x, x.y, x.z, x.w);
}
template <bool NT> __device__ inline uint2 ld_stream2(const uint16_t *p) {
  const u32x2_t *q = reinterpret_cast<const u32x2_t *>(p);
  u32x2_t x;
  if constexpr (NT) x = __builtin_nontemporal_load(q);
  else x = *q;
  return make_uint2(x.x, x.y);
}

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

// One piece of a workgroup's page range: pages [pbeg, pend) of KV head g of
// segment sg, whose partial goes to slot.
struct ItemPos {
  Seg sg;
  int g;        // KV head
  int pbeg;     // first page (segment-local)
  int pend;     // one past the last page
  int npages;   // pages in the segment
  int slot;     // partial slot
};

// A plain decode launch carries its plan in its arguments; a step launch
// reads it from device memory (scalar loads through the constant address
// space), so that its arguments stay the same from step to step.
#define SQ_CONST __attribute__((address_space(4)))
struct ArgPlan {
  const DecodeDyn &d;
  __device__ int n_segs() const { return d.n_segs; }
  __device__ int total() const { return d.total; }
  __device__ int n_wg() const { return d.n_wg; }
  __device__ int slot_base() const { return d.slot_base; }
  __device__ int row_pad() const { return d.row_pad; }
  __device__ bool masked() const { return d.masked != 0; }
  __device__ int seg_start(int i) const { return d.segs[i].start; }
  __device__ Seg seg(int i) const { return d.segs[i]; }
};
struct DevPlan {
  const SQ_CONST DecodeDyn *d;
  __device__ int n_segs() const { return d->n_segs; }
  __device__ int total() const { return d->total; }
  __device__ int n_wg() const { return d->n_wg; }
  __device__ int slot_base() const { return d->slot_base; }
  __device__ int row_pad() const { return d->row_pad; }
  __device__ bool masked() const { return d->masked != 0; }
  __device__ int seg_start(int i) const { return d->segs[i].start; }
  __device__ Seg seg(int i) const {
    const SQ_CONST Seg &x = d->segs[i];
    Seg y;
    y.page0 = x.page0;
    y.ntok = x.ntok;
    y.start = x.start;
    y.rmt = x.rmt;
    y.mem[0] = x.mem[0];
    y.mem[1] = x.mem[1];
    return y;
  }
};

// floor(w * total / n) for 0 <= w <= n <= kMaxItems and total < 2^31, in
// 32-bit arithmetic: with total = q n + r it is w q + floor(w r / n), and
// w r < 2^26.  (A 64-bit division is a long instruction sequence that every
// workgroup would run before its first load.)
__device__ inline int64_t split_point(int w, int total, int n) {
  const int q = total / n, r = total - q * n;
  return (int64_t)w * q + (w * r) / n;
}
static_assert(kMaxItems <= (1 << 13), "w r must stay below 2^26");

// The next piece of workgroup w's range [x, xe): the real pages of one row
// from x on (skipping row padding); advances x past it.  False when the
// range holds no more real pages.
template <class PL>
__device__ inline bool next_piece(const PL &pl, int hkv, int w, int64_t &x, int64_t xe, ItemPos &ip) {
  while (x < xe) {
    int lo = 0, hi = pl.n_segs() - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (pl.seg_start(mid) <= x) lo = mid;
      else hi = mid - 1;
    }
    ip.sg = pl.seg(lo);
    ip.npages = (ip.sg.ntok + P - 1) / P;
    const int64_t rl = ip.npages + pl.row_pad();
    ip.g = (int)(x - ip.sg.start) / (int)rl; // both below 2^31
    const int64_t rs = ip.sg.start + (int64_t)ip.g * rl;
    if (x - rs >= ip.npages) { // in the row's padding
      x = rs + rl;
      continue;
    }
    const int64_t pe = min(xe, rs + ip.npages);
    ip.pbeg = (int)(x - rs);
    ip.pend = (int)(pe - rs);
    ip.slot = pl.slot_base() + w + lo * hkv + ip.g;
    x = pe;
    return true;
  }
  return false;
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
template <int D, int G, bool NT, class PL, bool KV8 = false>
__device__ inline void valu_body(const DecodeStatic &a, const PL &pl) {
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
  if ((int)blockIdx.x >= pl.n_wg()) return;
  const int64_t x_end = split_point(blockIdx.x + 1, pl.total(), pl.n_wg());
  int64_t x_pos = split_point(blockIdx.x, pl.total(), pl.n_wg());
  ItemPos ip;
  while (next_piece(pl, a.hkv, blockIdx.x, x_pos, x_end, ip)) {
  const int b = ip.sg.member(0);
  const int g = ip.g;
  const int32_t *pt = a.pt + (int64_t)ip.sg.row() * a.max_pages + ip.sg.page0;
  const int32_t *mrow = a.mask + (int64_t)ip.sg.row() * a.max_pages + ip.sg.page0;
  const bool use_mask = pl.masked();

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

  // 8 elements per lane per load: 16 bytes of bf16, or 8 codes of an 8-bit
  // store converted to bf16 as they arrive (strides count elements)
  const uint16_t *kbase = a.k + (int64_t)g * a.head_stride + lane * 8;
  const uint16_t *vbase = a.v + (int64_t)g * a.head_stride + lane * 8;
  const uint8_t *kbase8 = reinterpret_cast<const uint8_t *>(a.k) + (int64_t)g * a.head_stride + lane * 8;
  const uint8_t *vbase8 = reinterpret_cast<const uint8_t *>(a.v) + (int64_t)g * a.head_stride + lane * 8;
  u32x4_t kreg[NLD], vreg[NLD];
  auto load_page = [&](int64_t off) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      if constexpr (KV8) {
        kreg[i] = ld_kv4_8<NT>(kbase8 + off + i * 512);
        vreg[i] = ld_kv4_8<NT>(vbase8 + off + i * 512);
      } else {
        kreg[i] = ld_kv4<NT>(kbase + off + i * 512);
        vreg[i] = ld_kv4<NT>(vbase + off + i * 512);
      }
    }
  };
  load_page((int64_t)pt[ip.pbeg] * a.page_stride);

  for (int pg = ip.pbeg; pg < ip.pend; ++pg) {
    const int valid = (pg == ip.npages - 1) ? ip.sg.ntok - pg * P : P;
    const int lo = pg == 0 ? ip.sg.tok0() : 0; // tokens before lo: outside a window
    // slots attended: [lo, valid) less those a deferred eviction masked
    const int live = (use_mask ? mrow[pg] : 0xffff) & ((1 << valid) - 1) & ~((1 << lo) - 1);
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
    if (pg + 1 < ip.pend) // prefetch the next page while this one is used
      load_page((int64_t)pt[pg + 1] * a.page_stride);

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
      x = ((live >> t) & 1) ? x * a.scale_log2 : kNegInf;
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
      if (valid < P || lo > 0) { // values of absent tokens may be anything: keep 0 * v finite
        v0 = 4 * R + 0 >= lo && 4 * R + 0 < valid ? v0 : 0.f;
        v1 = 4 * R + 1 >= lo && 4 * R + 1 < valid ? v1 : 0.f;
        v2 = 4 * R + 2 >= lo && 4 * R + 2 < valid ? v2 : 0.f;
        v3 = 4 * R + 3 >= lo && 4 * R + 3 < valid ? v3 : 0.f;
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

  const int64_t prow = (int64_t)ip.slot * kRows;
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
  __syncthreads();
  } // pieces
}

template <int D, int G, bool NT, bool KV8>
__global__ __launch_bounds__(64) void k_decode_valu(DecodeArgs a) {
  valu_body<D, G, NT, ArgPlan, KV8>(a.st, ArgPlan{a.dyn});
}
template <int D, int G, bool KV8>
__global__ __launch_bounds__(64) void k_step_valu(DecodeStatic a, const DecodeDyn *dyn) {
  valu_body<D, G, true, DevPlan, KV8>(a, DevPlan{(const SQ_CONST DecodeDyn *)dyn});
}

// ===========================================================================
// MFMA multi-query tile: up to 16 query rows (nmem sequences x G heads of one
// KV head) against the same pages.  A piece is processed by a workgroup of
// kWaves waves; wave w takes the w-th contiguous share of its pages and the
// waves' softmax states are combined in LDS at the end, so one piece still
// yields one partial per row.
// Lane l = n + 16 * kg (n = l & 15, kg = l >> 4):
//   QK A operand  K[token n][channels 8 kg + 32 s .. +8]       (16x16x32)
//   QK B operand  Q[row n][same channels]
//   S^T output    S[token 4 kg + i][row n], i < 4
//   PV A operand  V^T[channel n + 16 jd][tokens 4 kg .. +4]    (16x16x16)
//   PV B operand  P[row n][tokens 4 kg + i]  = the S^T registers after softmax
//   O^T output    O[row n][channel 16 jd + 4 kg + i]
// P is split into bf16 hi + lo parts (two MFMAs per block) so the weights
// keep ~16 bits; the running sum l uses the same hi + lo values.
template <int D> struct KFrag {
  uint4 k[D / 32];
};
template <int D> struct VFrag {
  uint2 v[D / 16];
};

// A buffer resource over one page of one KV head (the pools are read only
// through these): a page that is not wanted gets num_records 0, so its loads
// return zeros without touching memory and every loop iteration issues the
// same loads - which keeps the hardware's in-order load counter waits exact.
constexpr int kRsrcWord3 = 0x00020000;
__device__ inline __amdgpu_buffer_rsrc_t page_rsrc(const char *page, bool want, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(page), (short)0, want ? bytes : 0,
                                           kRsrcWord3);
}
template <bool NT> constexpr int kAux = NT ? 2 : 0; // nt: streamed once
// pages in flight per wave of the 8-bit MFMA tile (a 64-channel page is
// half the bytes, so twice as many keep the same bytes in flight)
template <int D> constexpr int kStages8 = D == 64 ? 4 : 2;
// waves per SIMD of the MFMA tiles
constexpr int kMfmaWavesPerEu = 3;

// K fragment: lane (n, kg) takes channels 8 kg + 32 s .. +8 of token n.
template <int D, bool NT>
__device__ inline void load_k(KFrag<D> &f, __amdgpu_buffer_rsrc_t r, int lane_off) {
#pragma unroll
  for (int s = 0; s < D / 32; ++s) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, lane_off + 64 * s, 0, kAux<NT>);
    f.k[s] = make_uint4(x[0], x[1], x[2], x[3]);
  }
}
// V^T fragment: lane (n, kg) takes tokens 4 kg .. +4 of channel n + 16 j.
template <int D, bool NT>
__device__ inline void load_v(VFrag<D> &f, __amdgpu_buffer_rsrc_t r, int lane_off) {
#pragma unroll
  for (int j = 0; j < D / 16; ++j) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b64(r, lane_off + 32 * P * j, 0, kAux<NT>);
    f.v[j] = make_uint2(x[0], x[1]);
  }
}

// The same fragments in an 8-bit store (E4M3 codes, half the bytes); they
// become bf16 fragments just before the matrix-core instructions.  A K lane
// loads 16 contiguous codes, channels 16 kg + 64 s' .. +16 of token n, in
// one request (a token's row is read in full-line halves, as in bf16); its
// two 8-channel halves feed QK chunks 2 s' and 2 s' + 1, and the query
// fragments take the same channels, so each chunk still pairs q and k
// channel by channel (the dot product is a sum over a permutation of the
// channels).
template <int D> struct KFrag8 {
  uint4 k[D / 64];
};
template <int D> struct VFrag8 {
  uint32_t v[D / 16];
};
template <int D, bool NT>
__device__ inline void load_k(KFrag8<D> &f, __amdgpu_buffer_rsrc_t r, int lane_off) {
#pragma unroll
  for (int s = 0; s < D / 64; ++s) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, lane_off + 64 * s, 0, kAux<NT>);
    f.k[s] = make_uint4(x[0], x[1], x[2], x[3]);
  }
}
// A V lane loads the 16 codes of one channel row, c = 64 J + 16 kg + n, in
// one request (four b32 requests would each carry 4 codes).  Word t of that
// row (tokens 4t .. 4t+3) belongs to the lane with the same n in lane row t,
// for matrix-core instruction 4 J + kg: a 4 x 4 transpose across the wave's
// four lane rows, done as the fragment is converted.
template <int D, bool NT>
__device__ inline void load_v(VFrag8<D> &f, __amdgpu_buffer_rsrc_t r, int lane_off) {
#pragma unroll
  for (int J = 0; J < D / 64; ++J) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, lane_off + 64 * P * J, 0, kAux<NT>);
#pragma unroll
    for (int t = 0; t < 4; ++t) f.v[4 * J + t] = x[t];
  }
}
template <int D> __device__ inline KFrag<D> to_bf16(const KFrag8<D> &f) {
  KFrag<D> o;
#pragma unroll
  for (int s = 0; s < D / 64; ++s) {
    const uint2 a = e4m3x4_to_bf16(f.k[s].x), b = e4m3x4_to_bf16(f.k[s].y);
    const uint2 c = e4m3x4_to_bf16(f.k[s].z), d = e4m3x4_to_bf16(f.k[s].w);
    o.k[2 * s] = make_uint4(a.x, a.y, b.x, b.y);
    o.k[2 * s + 1] = make_uint4(c.x, c.y, d.x, d.y);
  }
  return o;
}
template <int D, bool KV8> struct Frags {
  using K = KFrag<D>;
  using V = VFrag<D>;
};
template <int D> struct Frags<D, true> {
  using K = KFrag8<D>;
  using V = VFrag8<D>;
};
template <int D> __device__ inline const KFrag<D> &to_bf16(const KFrag<D> &f) { return f; }
template <int D> __device__ inline const VFrag<D> &to_bf16(const VFrag<D> &f) { return f; }
// Lane row r holds words w[0..3] of rows c = 64 J + 16 r + n; afterwards it
// holds word r of those rows for r' = 0..3.  Swapping lane rows {0,1} with
// {2,3} across word pairs (0,2) and (1,3) exchanges the off-diagonal 2 x 2
// blocks; swapping odd with even lane rows across pairs (0,1) and (2,3)
// transposes each block.
template <int D> __device__ inline VFrag<D> to_bf16(const VFrag8<D> &f) {
  VFrag<D> o;
#pragma unroll
  for (int J = 0; J < D / 64; ++J) {
    const auto a = __builtin_amdgcn_permlane32_swap(f.v[4 * J], f.v[4 * J + 2], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(f.v[4 * J + 1], f.v[4 * J + 3], false, false);
    const auto c = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
    const auto d = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
    o.v[4 * J] = e4m3x4_to_bf16(c[0]);
    o.v[4 * J + 1] = e4m3x4_to_bf16(c[1]);
    o.v[4 * J + 2] = e4m3x4_to_bf16(d[0]);
    o.v[4 * J + 3] = e4m3x4_to_bf16(d[1]);
  }
  return o;
}

// S^T = K . Q^T for one page, then the online-softmax update of (m, l, acc);
// returns the page's weights P as bf16 hi and lo parts.  Slots [lo, valid)
// are attended, and with MK only those whose bit is set in mk (the keep mask
// of deferred evictions).
template <int D, bool MK>
__device__ inline void mfma_scores(const KFrag<D> &f, int lo, int valid, int mk, int kg,
                                   float scale_log2,
                                   const bf16x8_t (&qb)[D / 32], f32x4_t (&acc)[D / 16],
                                   float &m_run, float &l_run, s16x4_t &phi, s16x4_t &plo) {
  constexpr int NS = D / 32;
  constexpr int NJ = D / 16;
  f32x4_t st = f32x4_t{0.f, 0.f, 0.f, 0.f};
  __builtin_amdgcn_s_setprio(1); // as in mfma_values
#pragma unroll
  for (int s = 0; s < NS; ++s)
    st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, f.k[s]), qb[s], st,
                                                 0, 0, 0);
  __builtin_amdgcn_s_setprio(0);
  float x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bool in = 4 * kg + i >= lo && 4 * kg + i < valid;
    if constexpr (MK) in = in && ((mk >> (4 * kg + i)) & 1);
    x[i] = in ? st[i] * scale_log2 : kNegInf;
  }
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
  phi = __builtin_bit_cast(s16x4_t, make_uint2(h01, h23));
  plo = __builtin_bit_cast(s16x4_t, make_uint2(l01, l23));
}

// O^T += V^T . P^T for one page (hi and lo parts of P).
template <int D>
__device__ inline void mfma_values(VFrag<D> &f, int lo, int valid, int kg, s16x4_t phi,
                                   s16x4_t plo, f32x4_t (&acc)[D / 16]) {
  constexpr int NJ = D / 16;
  if (valid < P || lo > 0) { // values of absent tokens may be anything: keep 0 * v finite
    auto in = [&](int t) { return t >= lo && t < valid; };
    const uint32_t m0 = (in(4 * kg + 0) ? 0xffffu : 0u) | (in(4 * kg + 1) ? 0xffff0000u : 0u);
    const uint32_t m1 = (in(4 * kg + 2) ? 0xffffu : 0u) | (in(4 * kg + 3) ? 0xffff0000u : 0u);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      f.v[j].x &= m0;
      f.v[j].y &= m1;
    }
  }
  // raised priority while the MFMAs issue lets the other waves' VALU work
  // interleave with them (measured: about 0.5% on the 128K shared-prefix step)
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const s16x4_t vA = __builtin_bit_cast(s16x4_t, f.v[j]);
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vA, phi, acc[j], 0, 0, 0);
    acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vA, plo, acc[j], 0, 0, 0);
  }
  __builtin_amdgcn_s_setprio(0);
}

// MK: the plan may carry keep masks (decided at run time by the plan; false
// compiles the mask path out).  KV8: the pools hold E4M3 codes.  RB: row
// blocks of 16 query rows per tile; with RB = 2 the second block (rows
// 16..31: the members past 16 / G of a wide tile) takes the same K and V
// fragments of each page through its own matrix-core instructions, and a
// piece writes two consecutive partial slots.
template <int D, int G, int kWaves, bool NT, bool MK, class PL, bool KV8 = false, int RB = 1>
__device__ inline void mfma_body(const DecodeStatic &a, const PL &pl) {
  static_assert(RB == 1 || (RB == 2 && !KV8), "two row blocks on bf16 stores only");
  constexpr int NS = D / 32;
  constexpr int NJ = D / 16;
  constexpr int APITCH = D + 4; // floats per row of a wave's accumulator in LDS
  __shared__ float s_m[kWaves][kRows];
  __shared__ float s_l[kWaves][kRows];
  __shared__ __attribute__((aligned(16))) float s_acc[kWaves][kRows * APITCH];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); // uniform in the wave
  const int n = lane & 15, kg = lane >> 4;
  if ((int)blockIdx.x >= pl.n_wg()) return;
  const int64_t x_end = split_point(blockIdx.x + 1, pl.total(), pl.n_wg());
  int64_t x_pos = split_point(blockIdx.x, pl.total(), pl.n_wg());
  ItemPos ip;
  while (next_piece(pl, a.hkv, blockIdx.x, x_pos, x_end, ip)) {
  const int g = ip.g;
  const int nrows = ip.sg.nmem() * G;
  const bool two = RB > 1 && nrows > kRows; // uniform: the piece uses block 1
  const int32_t *pt = a.pt + (int64_t)ip.sg.row() * a.max_pages + ip.sg.page0;

  bf16x8_t qb[RB][NS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int row = n + kRows * rb;
    const bool qvalid = row < nrows;
    const int jm = qvalid ? row / G : 0;
    const int bq = ip.sg.member(jm);
    const uint16_t *qp = a.q + ((int64_t)bq * a.hq + g * G + row % G) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      // rows past nrows read member 0's row (in bounds) and are zeroed; an
      // 8-bit store's chunk s takes the channels its K fragments hold
      const int c0 = KV8 ? 16 * kg + 64 * (s >> 1) + 8 * (s & 1) : 8 * kg + 32 * s;
      uint4 w = *reinterpret_cast<const uint4 *>(qp + c0);
      if (!qvalid) w = make_uint4(0, 0, 0, 0);
      qb[rb][s] = __builtin_bit_cast(bf16x8_t, w);
    }
  }

  f32x4_t acc[RB][NJ];
  float m_run[RB], l_run[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[rb][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    m_run[rb] = kNegInf;
    l_run[rb] = 0.f;
  }

  constexpr int ES = KV8 ? 1 : 2; // bytes per element
  const char *khead = reinterpret_cast<const char *>(a.k) + (int64_t)g * a.head_stride * ES;
  const char *vhead = reinterpret_cast<const char *>(a.v) + (int64_t)g * a.head_stride * ES;
  const int koff = KV8 ? n * D + 16 * kg : (n * D + 8 * kg) * ES; // byte offsets within a page
  const int voff = KV8 ? (16 * kg + n) * P : (n * P + 4 * kg) * ES;
  constexpr int kPageBytes = P * D * ES;
  // Wave w takes the w-th of kWaves contiguous shares of the piece's pages.
  // Two pages are in flight while one is computed: page j + 2's K is loaded
  // into page j's K registers as soon as its scores are taken, and its V
  // into page j's V registers after the values, so every load has two
  // pages' worth of time to land.  Every iteration issues the same loads
  // (a page past the end gets an empty buffer and reads zeros), so the waits
  // on the in-order vector load counter stay exact.  Page ids are scalar
  // loads (their own counter), fetched an iteration before they are needed.
  const int np_piece = ip.pend - ip.pbeg;
  const int wbeg = ip.pbeg + np_piece * wave / kWaves;
  const int count = ip.pbeg + np_piece * (wave + 1) / kWaves - wbeg;
  typedef const int32_t __attribute__((address_space(4))) *sptr_t;
  const sptr_t ids = (sptr_t)(pt + wbeg);
  auto sid = [&](int j) -> int { return ids[min(j, max(count - 1, 0))]; };
  auto rsrc = [&](const char *head, int id, bool want) {
    return page_rsrc(head + (int64_t)(want ? id : 0) * a.page_stride * ES, want, kPageBytes);
  };
  auto valid_of = [&](int j) -> int {
    const int pg = wbeg + j;
    return j >= count ? 0 : (pg == ip.npages - 1) ? ip.sg.ntok - pg * P : P;
  };
  auto lo_of = [&](int j) -> int { return wbeg + j == 0 ? ip.sg.tok0() : 0; };
  // keep masks of deferred evictions, scalar loads like the ids (all ones
  // when the plan has none)
  const bool use_mask = MK && pl.masked();
  const sptr_t mids =
      (sptr_t)(a.mask + (int64_t)ip.sg.row() * a.max_pages + ip.sg.page0 + wbeg);
  auto smask = [&](int j) -> int { return use_mask ? mids[min(j, max(count - 1, 0))] : 0xffff; };
  if constexpr (KV8 && kStages8<D> > 2) {
  // An 8-bit page is half the bytes: more pages in flight, the same scheme
  // in arrays.
  constexpr int NST = kStages8<D>;
  KFrag8<D> kf[NST];
  VFrag8<D> vf[NST];
  int nid[NST], mkc[NST], mkn[NST]; // ids and masks of pages j + NST + st; masks in flight
  if (count > 0) {
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const int id = sid(st);
      load_k<D, NT>(kf[st], rsrc(khead, id, st == 0 || st < count), koff);
      load_v<D, NT>(vf[st], rsrc(vhead, id, st == 0 || st < count), voff);
      mkc[st] = smask(st);
    }
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      nid[st] = sid(NST + st);
      mkn[st] = smask(NST + st);
    }
  }
  for (int j = 0; j < count; j += NST) {
    // pages past count have zero fragments and no valid token: the update
    // leaves (m, l, acc) as they are
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const int valid = valid_of(j + st), lo = lo_of(j + st);
      s16x4_t phi, plo;
      mfma_scores<D, MK>(to_bf16(kf[st]), lo, valid, mkc[st], kg, a.scale_log2, qb[0], acc[0],
                         m_run[0], l_run[0], phi, plo);
      load_k<D, NT>(kf[st], rsrc(khead, nid[st], j + NST + st < count), koff);
      VFrag<D> vb = to_bf16(vf[st]);
      mfma_values<D>(vb, lo, valid, kg, phi, plo, acc[0]);
      load_v<D, NT>(vf[st], rsrc(vhead, nid[st], j + NST + st < count), voff);
      mkc[st] = mkn[st];
    }
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      nid[st] = sid(j + 2 * NST + st);
      mkn[st] = smask(j + 2 * NST + st);
    }
  }
  } else {
  typename Frags<D, KV8>::K k0, k1;
  typename Frags<D, KV8>::V v0, v1;
  int n0 = 0, n1 = 0;   // ids of pages j + 2 and j + 3
  int mk0 = 0, mk1 = 0; // masks of pages j and j + 1 (in the fragments)
  int q0 = 0, q1 = 0;   // masks of pages j + 2 and j + 3
  if (count > 0) {
    const int i0 = sid(0), i1 = sid(1);
    load_k<D, NT>(k0, rsrc(khead, i0, true), koff);
    load_v<D, NT>(v0, rsrc(vhead, i0, true), voff);
    load_k<D, NT>(k1, rsrc(khead, i1, count > 1), koff);
    load_v<D, NT>(v1, rsrc(vhead, i1, count > 1), voff);
    n0 = sid(2);
    n1 = sid(3);
    mk0 = smask(0);
    mk1 = smask(1);
    q0 = smask(2);
    q1 = smask(3);
  }
  for (int j = 0; j < count; j += 2) {
    {
      const int valid = valid_of(j), lo = lo_of(j);
      s16x4_t phi[RB], plo[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb == 0 || two)
          mfma_scores<D, MK>(to_bf16(k0), lo, valid, mk0, kg, a.scale_log2, qb[rb], acc[rb],
                             m_run[rb], l_run[rb], phi[rb], plo[rb]);
      load_k<D, NT>(k0, rsrc(khead, n0, j + 2 < count), koff);
      VFrag<D> vb0 = to_bf16(v0);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb == 0 || two) mfma_values<D>(vb0, lo, valid, kg, phi[rb], plo[rb], acc[rb]);
      load_v<D, NT>(v0, rsrc(vhead, n0, j + 2 < count), voff);
      mk0 = q0;
    }
    {
      // page j + 1 may not exist (count odd): its fragments are then zeros
      // and with no valid token the update leaves (m, l, acc) as they are.
      const int valid = valid_of(j + 1), lo = lo_of(j + 1);
      s16x4_t phi[RB], plo[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb == 0 || two)
          mfma_scores<D, MK>(to_bf16(k1), lo, valid, mk1, kg, a.scale_log2, qb[rb], acc[rb],
                             m_run[rb], l_run[rb], phi[rb], plo[rb]);
      load_k<D, NT>(k1, rsrc(khead, n1, j + 3 < count), koff);
      VFrag<D> vb1 = to_bf16(v1);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (rb == 0 || two) mfma_values<D>(vb1, lo, valid, kg, phi[rb], plo[rb], acc[rb]);
      load_v<D, NT>(v1, rsrc(vhead, n1, j + 3 < count), voff);
      mk1 = q1;
    }
    n0 = sid(j + 4);
    n1 = sid(j + 5);
    q0 = smask(j + 4);
    q1 = smask(j + 5);
  }

  }

  // combine the waves' states: M = max m_w, scale_w = 2^(m_w - M).  The
  // thread index is re-read here so that the LDS addresses below are
  // computed after the page loop instead of being held through it.
  int tx = threadIdx.x;
  __asm__ volatile("" : "+v"(tx));
  const int ew = tx >> 6, en = tx & 15, ekg = (tx >> 4) & 3;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
  if (rb > 0 && !two) break;
  if (rb > 0) __syncthreads(); // the previous block's combination has read the LDS
  float l_tot = sum_xrow16(l_run[rb]);
  l_tot = sum_xrow32(l_tot);
  if (ekg == 0) {
    s_m[ew][en] = m_run[rb];
    s_l[ew][en] = l_tot;
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    *reinterpret_cast<float4 *>(&s_acc[ew][en * APITCH + 16 * j + 4 * ekg]) =
        make_float4(acc[rb][j][0], acc[rb][j][1], acc[rb][j][2], acc[rb][j][3]);
  __syncthreads();
  // a piece's RB slots are consecutive: slot_base + RB * (its index) + rb
  const int64_t prow =
      ((int64_t)pl.slot_base() + (int64_t)RB * (ip.slot - pl.slot_base()) + rb) * kRows;
  const int nr = nrows - kRows * rb; // rows of this block
  if (tx < kRows && tx < nr) {
    const int r = tx;
    float mm = kNegInf;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mm = fmaxf(mm, s_m[w][r]);
    float ll = 0.f;
    if (mm != kNegInf) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) ll += exp2_fast(s_m[w][r] - mm) * s_l[w][r];
    }
    a.part_m[prow + r] = mm;
    a.part_l[prow + r] = ll;
  }
  constexpr int PER = kRows * D / (64 * kWaves); // output floats per thread
  const int e0 = tx * PER;
  const int r = e0 / D;
  if (r < nr) {
    float mm = kNegInf;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mm = fmaxf(mm, s_m[w][r]);
    float sc[kWaves];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) sc[w] = mm == kNegInf ? 0.f : exp2_fast(s_m[w][r] - mm);
    const int d0 = e0 % D;
#pragma unroll
    for (int e = 0; e < PER; e += 4) {
      float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float4 x = *reinterpret_cast<const float4 *>(&s_acc[w][r * APITCH + d0 + e]);
        o.x = fmaf(sc[w], x.x, o.x);
        o.y = fmaf(sc[w], x.y, o.y);
        o.z = fmaf(sc[w], x.z, o.z);
        o.w = fmaf(sc[w], x.w, o.w);
      }
      *reinterpret_cast<float4 *>(a.part_acc + (prow + r) * D + d0 + e) = o;
    }
  }
  } // row blocks
  __syncthreads(); // the next piece reuses the LDS
  } // pieces
}

template <int D, int G, int kWaves, bool NT, bool MK>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(kMfmaWavesPerEu, kMfmaWavesPerEu))) void
k_decode_mfma(DecodeArgs a) {
  mfma_body<D, G, kWaves, NT, MK>(a.st, ArgPlan{a.dyn});
}
// Two row blocks (wide tiles of a tree's shared runs): twice the
// accumulators, two waves per SIMD.
template <int D, int G, int kWaves, bool NT, bool MK>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2))) void
k_decode_mfma2(DecodeArgs a) {
  mfma_body<D, G, kWaves, NT, MK, ArgPlan, false, 2>(a.st, ArgPlan{a.dyn});
}
template <int D, int G, int kWaves>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(kMfmaWavesPerEu, kMfmaWavesPerEu))) void
k_step_mfma(DecodeStatic a, const DecodeDyn *dyn) {
  mfma_body<D, G, kWaves, true, true>(a, DevPlan{(const SQ_CONST DecodeDyn *)dyn});
}
// 8-bit store: four waves, streaming loads
template <int D, int G, bool MK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kMfmaWavesPerEu, kMfmaWavesPerEu))) void
k_decode_mfma8(DecodeArgs a) {
  mfma_body<D, G, 4, true, MK, ArgPlan, true>(a.st, ArgPlan{a.dyn});
}
template <int D, int G>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(kMfmaWavesPerEu, kMfmaWavesPerEu))) void
k_step_mfma8(DecodeStatic a, const DecodeDyn *dyn) {
  mfma_body<D, G, 4, true, true, DevPlan, true>(a, DevPlan{(const SQ_CONST DecodeDyn *)dyn});
}

// ===========================================================================
// Merge: one workgroup of kMergeWaves waves per (batch entry, query head).
// Its partials are the pieces of at most kMaxSrc segments (the shared runs on
// its path through the tree of forks, then its own suffix).  Thread t takes
// channel t % D of share t / D of each round of NSH * kMergeChunk pieces
// (the round's partial rows listed in LDS first, pieces dealt to the shares
// round-robin): it loads its share's
// (m, l) pairs itself (the same addresses across the share's threads, one
// request per wave) and its channel of each acc row, all in flight
// together, and folds them into a running (m, l, acc) with the usual
// rescale.  No cross-lane reduction; the shares (and the sink, and in a
// step the new token) combine through LDS.  Latency, not bandwidth, bounds
// this kernel: one round of loads covers a (batch entry, head)'s pieces
// when there are at most NSH * kMergeChunk of them.
constexpr int kMergeWaves = 8;
constexpr int kMergeChunk = 24;

struct ArgMerge {
  const MergeDyn &d;
  __device__ int total(int L) const { return d.total[L]; }
  __device__ int n_wg(int L) const { return d.n_wg[L]; }
  __device__ int slot_base(int L) const { return d.slot_base[L]; }
  __device__ int row_pad(int L) const { return d.row_pad[L]; }
  __device__ int n_src(int b) const { return d.n_src[b]; }
  __device__ int rb(int L) const { return d.rb[L]; }
  __device__ int src(int b, int e) const { return (int)((d.src[b][e >> 1] >> (16 * (e & 1))) & 0xffff); }
  __device__ int seg_start(int i) const { return d.seg_start[i]; }
  __device__ int seg_npages(int i) const { return d.seg_npages[i]; }
  __device__ int seg_meta(int i) const { return d.seg_meta[i]; }
};
struct DevMerge {
  const SQ_CONST MergeDyn *d;
  __device__ int total(int L) const { return d->total[L]; }
  __device__ int n_wg(int L) const { return d->n_wg[L]; }
  __device__ int slot_base(int L) const { return d->slot_base[L]; }
  __device__ int row_pad(int L) const { return d->row_pad[L]; }
  __device__ int n_src(int b) const { return d->n_src[b]; }
  __device__ int rb(int L) const { return d->rb[L]; }
  __device__ int src(int b, int e) const { return (int)((d->src[b][e >> 1] >> (16 * (e & 1))) & 0xffff); }
  __device__ int seg_start(int i) const { return d->seg_start[i]; }
  __device__ int seg_npages(int i) const { return d->seg_npages[i]; }
  __device__ int seg_meta(int i) const { return d->seg_meta[i]; }
};

// With APPEND (a decode step), the entry's new token is one more term -
// score q . k_new, weight 1, value v_new - and the workgroup of the first
// query head of each KV head stores the new token's K, V and position for
// later steps.  KV8 (with APPEND): the new token is stored as E4M3 codes and
// joins the softmax as stored (its codes; the K scale is in scale_log2, the
// V scale in out_scale).
// The grid is (G, Hkv, batch): workgroup (hr, g, b) merges query head
// g * G + hr of batch entry b.  With has_inl, rows holds that (b, g)'s row
// lists (the call carries them in its arguments); else they are derived
// from the plan.
template <int D, bool APPEND, class MP, class SA, bool KV8 = false>
__device__ inline void merge_body(const MergeStatic &a, const MP &mp, const SA &sa, bool has_inl,
                                  const MergeRows &rows) {
  constexpr int NT = 64 * kMergeWaves;
  constexpr int NSH = NT / D; // piece shares
  constexpr int NX = NSH + 2; // the shares, then the sink, then the new token
  constexpr int CH = kMergeChunk;
  static_assert(NT % D == 0 && D % 64 == 0, "whole waves per share");
  __shared__ float s_m[NX];
  __shared__ float s_l[NX];
  __shared__ float s_a[NX][D];
  __shared__ float s_dot[D / 64];
  const int tid = threadIdx.x;
  const int c = tid % D, sh = tid / D;
  const int hr = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int h = g * (int)gridDim.x + hr;
  int cum[kMaxSrc + 1];
  int32_t base[kMaxSrc], step[kMaxSrc];
  cum[0] = 0;
  // (read before the test, so that they come in the first round of
  // argument reads whichever way it goes)
  int32_t ib[kMaxSrc], ics[kMaxSrc];
#pragma unroll
  for (int e = 0; e < kMaxSrc; ++e) {
    ib[e] = rows.base[e];
    ics[e] = rows.cnt_step[e];
    __asm__ volatile("" ::"s"(ib[e]), "s"(ics[e]));
  }
  if (has_inl) {
#pragma unroll
    for (int e = 0; e < kMaxSrc; ++e) {
      const uint32_t cs = (uint32_t)ics[e];
      base[e] = ib[e] + hr;
      step[e] = (int)(cs >> 16);
      cum[e + 1] = cum[e] + (int)(cs & 0xffff);
    }
  } else {
  const int ns = mp.n_src(b);
#pragma unroll
  for (int e = 0; e < kMaxSrc; ++e) {
    int cnt = 0;
    base[e] = 0;
    step[e] = kRows;
    if (e < ns) {
      const int sr = mp.src(b, e);
      const int si = sr & 0xff, member = (sr >> 8) & 0xf;
      const int meta = mp.seg_meta(si);
      const int L = meta & 1, seg = meta >> 1;
      const int np = mp.seg_npages(si);
      const int64_t R = (int64_t)mp.seg_start(si) + (int64_t)g * (np + mp.row_pad(L)); // row start
      const int w_lo = wg_of(R, mp.total(L), mp.n_wg(L));
      const int w_hi = wg_of(R + np - 1, mp.total(L), mp.n_wg(L));
      cnt = w_hi - w_lo + 1;
      // a piece of an RB-block launch owns RB consecutive slots of 16 rows
      step[e] = mp.rb(L) * kRows;
      base[e] = (mp.slot_base(L) + mp.rb(L) * (w_lo + seg * a.hkv + g)) * kRows +
                member * a.group + hr;
    }
    cum[e + 1] = cum[e] + cnt;
  }
  } // row lists from the plan
  const int total = cum[kMaxSrc];
  auto row_of = [&](int i) -> int32_t {
    int e = 0;
#pragma unroll
    for (int k = 1; k < kMaxSrc; ++k) e += i >= cum[k];
    return base[e] + (i - cum[e]) * step[e];
  };

  // rounds of TILE pieces: the workgroup first lists the round's partial
  // rows in LDS (one row lookup per thread), then share sh folds pieces
  // sh, sh + NSH, ... of the round (pieces dealt round-robin, so that a few
  // pieces still spread over every share), all of their loads in flight
  // together
  constexpr int TILE = NSH * CH;
  static_assert(TILE <= NT, "one row per thread and round");
  __shared__ int32_t s_rows[TILE];
  float m_r = kNegInf, l_r = 0.f, a_r = 0.f;
  for (int t0 = 0; t0 < total; t0 += TILE) {
    const int nt = min(TILE, total - t0);
    if (tid < nt) s_rows[tid] = row_of(t0 + tid);
    __syncthreads();
    const int cnt = sh < nt ? (nt - sh + NSH - 1) / NSH : 0; // this share's pieces (uniform)
    float mv[CH], lv[CH], av[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      mv[u] = kNegInf;
      lv[u] = 0.f;
      av[u] = 0.f;
      if (u < cnt) {
        const int32_t row = s_rows[sh + NSH * u];
        mv[u] = a.part_m[row];
        lv[u] = a.part_l[row];
        av[u] = a.part_acc[(int64_t)row * D + c];
      }
    }
    float mx = m_r;
#pragma unroll
    for (int u = 0; u < CH; ++u) mx = fmaxf(mx, mv[u]);
    if (mx != kNegInf) { // else only empty pieces so far
      const float sc = exp2_fast(m_r - mx); // 0 while m_r is -inf
      l_r *= sc;
      a_r *= sc;
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const float w = exp2_fast(mv[u] - mx); // 0 for empty and absent pieces
        l_r = fmaf(w, lv[u], l_r);
        a_r = fmaf(w, av[u], a_r);
      }
      m_r = mx;
    }
    __syncthreads(); // s_rows is rewritten next round
  }
  if (c == 0) {
    s_m[sh] = m_r;
    s_l[sh] = l_r;
  }
  s_a[sh][c] = a_r;
  if (sh == NSH - 1) { // the extra terms: the sink (no value), the new token
    s_a[NSH][c] = 0.f;
    float vnew = 0.f;
    if constexpr (APPEND) {
      const int64_t kv = (int64_t)b * a.hkv + g;
      const uint16_t kraw = sa.k_new[kv * D + c], vraw = sa.v_new[kv * D + c];
      float kf = __uint_as_float((uint32_t)kraw << 16), vf = __uint_as_float((uint32_t)vraw << 16);
      uint16_t kb = kraw, vb = vraw;
      if constexpr (KV8) { // the codes, and their values as the store holds them
        kb = (uint16_t)e4m3_encode(kf * sa.inv_k);
        vb = (uint16_t)e4m3_encode(vf * sa.inv_v);
        kf = __uint_as_float(e4m3x4_to_bf16(kb).x << 16);
        vf = __uint_as_float(e4m3x4_to_bf16(vb).x << 16);
      }
      float dot = __uint_as_float((uint32_t)sa.q[((int64_t)b * a.hq + h) * D + c] << 16) * kf;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
      if ((tid & 63) == 0) s_dot[(tid >> 6) % (D / 64)] = dot;
      vnew = vf;
      if (hr == 0) { // store the new token of KV head g (the same in every head's workgroup)
        const SQ_CONST StepAppend &ap = ((const SQ_CONST StepPlan *)sa.plan)->app;
        const int page = ap.page[b], slot = ap.slot[b];
        const int64_t pb = (int64_t)g * sa.head_stride + (int64_t)page * sa.page_stride;
        if constexpr (KV8) {
          uint8_t *k8 = reinterpret_cast<uint8_t *>(sa.k), *v8 = reinterpret_cast<uint8_t *>(sa.v);
          k8[pb + (int64_t)slot * D + c] = (uint8_t)kb;
          v8[pb + (int64_t)c * P + slot] = (uint8_t)vb;
        } else {
          sa.k[pb + (int64_t)slot * D + c] = kb;
          sa.v[pb + (int64_t)c * P + slot] = vb;
        }
        if (c == 0 && g == 0) sa.pos[(int64_t)page * P + slot] = ap.pos[b];
      }
    }
    s_a[NSH + 1][c] = vnew;
  }
  __syncthreads();
  if (tid < D) {
    float xm[NX], xl[NX];
#pragma unroll
    for (int x = 0; x < NSH; ++x) {
      xm[x] = s_m[x];
      xl[x] = s_l[x];
    }
    xm[NSH] = a.sinks ? a.sinks[h] * a.sink_scale : kNegInf;
    xl[NSH] = a.sinks ? 1.f : 0.f;
    xm[NSH + 1] = kNegInf;
    xl[NSH + 1] = 0.f;
    if constexpr (APPEND) {
      float dot = 0.f;
#pragma unroll
      for (int w = 0; w < D / 64; ++w) dot += s_dot[w];
      xm[NSH + 1] = dot * sa.scale_log2;
      xl[NSH + 1] = 1.f;
    }
    float mm = kNegInf;
#pragma unroll
    for (int x = 0; x < NX; ++x) mm = fmaxf(mm, xm[x]);
    float num = 0.f, den = 0.f;
    if (mm != kNegInf) {
#pragma unroll
      for (int x = 0; x < NX; ++x) {
        const float w = exp2_fast(xm[x] - mm); // 0 for -inf terms
        den = fmaf(w, xl[x], den);
        num = fmaf(w, s_a[x][c], num);
      }
    }
    a.out[((int64_t)b * a.hq + h) * D + c] = den > 0.f ? num / den * a.out_scale : 0.f;
  }
}

__constant__ MergeRows kNoRows = {}; // step merges derive their row lists from the plan

template <int D>
__global__ __launch_bounds__(64 * kMergeWaves) void k_decode_merge(MergeArgs a) {
  // (from the workgroup's own ids: no argument read before this one)
  const int bg = min((int)(blockIdx.z * kInlineG + blockIdx.y), kInlineRows - 1);
  merge_body<D, false>(a.st, ArgMerge{a.dyn}, 0, a.n_inline != 0, a.rows[bg]);
}
template <int D>
__global__ __launch_bounds__(64 * kMergeWaves) void k_step_merge(StepMergeArgs a) {
  const SQ_CONST StepPlan *plan = (const SQ_CONST StepPlan *)a.plan;
  if ((int)blockIdx.z >= plan->batch) return; // a replay sized for a larger batch
  merge_body<D, true>(a.st, DevMerge{a.windowed ? &plan->merge_w : &plan->merge}, a, false, kNoRows);
}
template <int D> __global__ __launch_bounds__(64 * kMergeWaves) void k_step_merge8(StepMergeArgs a) {
  const SQ_CONST StepPlan *plan = (const SQ_CONST StepPlan *)a.plan;
  if ((int)blockIdx.z >= plan->batch) return;
  merge_body<D, true, DevMerge, StepMergeArgs, true>(
      a.st, DevMerge{a.windowed ? &plan->merge_w : &plan->merge}, a, false, kNoRows);
}

template <int D, bool NT, bool KV8>
hipError_t valu_dispatch_nt(int group, const DecodeArgs &a, hipStream_t s) {
  const dim3 grid(a.dyn.n_wg), block(64);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_decode_valu<D, 1, NT, KV8>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_decode_valu<D, 2, NT, KV8>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_valu<D, 4, NT, KV8>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_valu<D, 8, NT, KV8>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D>
hipError_t valu_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  if (a.st.kv8)
    return a.st.nontemporal ? valu_dispatch_nt<D, true, true>(group, a, s)
                            : valu_dispatch_nt<D, false, true>(group, a, s);
  return a.st.nontemporal ? valu_dispatch_nt<D, true, false>(group, a, s)
                       : valu_dispatch_nt<D, false, false>(group, a, s);
}

template <int D, int W, bool NT, bool MK>
hipError_t mfma_dispatch_w(int group, const DecodeArgs &a, hipStream_t s) {
  const dim3 grid(a.dyn.n_wg), block(64 * W);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_decode_mfma<D, 1, W, NT, MK>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_decode_mfma<D, 2, W, NT, MK>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_mfma<D, 4, W, NT, MK>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_mfma<D, 8, W, NT, MK>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D, bool MK>
hipError_t mfma8_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  const dim3 grid(a.dyn.n_wg), block(256);
  switch (group) {
  case 1: hipLaunchKernelGGL((k_decode_mfma8<D, 1, MK>), grid, block, 0, s, a); break;
  case 2: hipLaunchKernelGGL((k_decode_mfma8<D, 2, MK>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_mfma8<D, 4, MK>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_mfma8<D, 8, MK>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D, bool NT, bool MK>
hipError_t mfma2_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  constexpr int W = kMfmaWaves;
  const dim3 grid(a.dyn.n_wg), block(64 * W);
  switch (group) { // G = 1 never needs a second block (at most 8 members)
  case 2: hipLaunchKernelGGL((k_decode_mfma2<D, 2, W, NT, MK>), grid, block, 0, s, a); break;
  case 4: hipLaunchKernelGGL((k_decode_mfma2<D, 4, W, NT, MK>), grid, block, 0, s, a); break;
  case 8: hipLaunchKernelGGL((k_decode_mfma2<D, 8, W, NT, MK>), grid, block, 0, s, a); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// a plan with keep masks takes the masked variant (ordinary loads); an
// 8-bit store its own kernel (four waves); tiles wider than 16 query rows
// the two-block kernel
template <int D>
hipError_t mfma_dispatch(int group, const DecodeArgs &a, hipStream_t s) {
  if (a.st.kv8) {
    if (a.dyn.rb != 1) return hipErrorInvalidValue;
    return a.dyn.masked ? mfma8_dispatch<D, true>(group, a, s) : mfma8_dispatch<D, false>(group, a, s);
  }
  if (a.dyn.rb == 2) {
    if (a.dyn.masked) return mfma2_dispatch<D, false, true>(group, a, s);
    return a.st.nontemporal ? mfma2_dispatch<D, true, false>(group, a, s)
                            : mfma2_dispatch<D, false, false>(group, a, s);
  }
  if (a.dyn.rb != 1) return hipErrorInvalidValue;
  if (a.dyn.masked) return mfma_dispatch_w<D, kMfmaWaves, false, true>(group, a, s);
  return a.st.nontemporal ? mfma_dispatch_w<D, kMfmaWaves, true, false>(group, a, s)
                       : mfma_dispatch_w<D, kMfmaWaves, false, false>(group, a, s);
}

} // namespace

namespace {
template <int D, bool KV8> const void *valu_fn(int group) {
  switch (group) {
  case 1: return reinterpret_cast<const void *>(&k_decode_valu<D, 1, true, KV8>);
  case 2: return reinterpret_cast<const void *>(&k_decode_valu<D, 2, true, KV8>);
  case 4: return reinterpret_cast<const void *>(&k_decode_valu<D, 4, true, KV8>);
  case 8: return reinterpret_cast<const void *>(&k_decode_valu<D, 8, true, KV8>);
  default: return nullptr;
  }
}
template <int D, int W> const void *mfma_fn_w(int group) {
  switch (group) {
  case 1: return reinterpret_cast<const void *>(&k_decode_mfma<D, 1, W, true, false>);
  case 2: return reinterpret_cast<const void *>(&k_decode_mfma<D, 2, W, true, false>);
  case 4: return reinterpret_cast<const void *>(&k_decode_mfma<D, 4, W, true, false>);
  case 8: return reinterpret_cast<const void *>(&k_decode_mfma<D, 8, W, true, false>);
  default: return nullptr;
  }
}
template <int D> const void *mfma8_fn(int group) {
  switch (group) {
  case 1: return reinterpret_cast<const void *>(&k_decode_mfma8<D, 1, false>);
  case 2: return reinterpret_cast<const void *>(&k_decode_mfma8<D, 2, false>);
  case 4: return reinterpret_cast<const void *>(&k_decode_mfma8<D, 4, false>);
  case 8: return reinterpret_cast<const void *>(&k_decode_mfma8<D, 8, false>);
  default: return nullptr;
  }
}
template <int D> const void *mfma_fn(int group) { return mfma_fn_w<D, kMfmaWaves>(group); }
template <int D> const void *mfma2_fn(int group) {
  switch (group) {
  case 2: return reinterpret_cast<const void *>(&k_decode_mfma2<D, 2, kMfmaWaves, true, false>);
  case 4: return reinterpret_cast<const void *>(&k_decode_mfma2<D, 4, kMfmaWaves, true, false>);
  case 8: return reinterpret_cast<const void *>(&k_decode_mfma2<D, 8, kMfmaWaves, true, false>);
  default: return nullptr;
  }
}
} // namespace

hipError_t decode_blocks_per_cu(int kind, int d, int group, int *out) {
  const void *fn = kind == 0   ? (d == 128 ? valu_fn<128, false>(group) : valu_fn<64, false>(group))
                   : kind == 3 ? (d == 128 ? valu_fn<128, true>(group) : valu_fn<64, true>(group))
                   : kind == 2 ? (d == 128 ? mfma8_fn<128>(group) : mfma8_fn<64>(group))
                   : kind == 4 ? (d == 128 ? mfma2_fn<128>(group) : mfma2_fn<64>(group))
                               : (d == 128 ? mfma_fn<128>(group) : mfma_fn<64>(group));
  if (!fn) return hipErrorInvalidValue;
  const int block = kind == 0 || kind == 3 ? 64 : 64 * kMfmaWaves;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(out, fn, block, 0);
}

hipError_t launch_decode_valu(int d, int group, const DecodeArgs &a, hipStream_t s) {
  if (a.dyn.n_wg == 0) return hipSuccess;
  return d == 128 ? valu_dispatch<128>(group, a, s) : valu_dispatch<64>(group, a, s);
}

hipError_t launch_decode_mfma(int d, int group, const DecodeArgs &a, hipStream_t s) {
  if (a.dyn.n_wg == 0) return hipSuccess;
  return d == 128 ? mfma_dispatch<128>(group, a, s) : mfma_dispatch<64>(group, a, s);
}

hipError_t launch_decode_merge(int d, int batch, const MergeArgs &a, hipStream_t s) {
  const dim3 grid(a.st.group, a.st.hkv, batch), block(64 * kMergeWaves);
  if (d == 128)
    hipLaunchKernelGGL(k_decode_merge<128>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_decode_merge<64>, grid, block, 0, s, a);
  return hipGetLastError();
}

namespace {
template <int D>
hipError_t step_valu_dispatch(int group, const DecodeStatic &st, const DecodeDyn *dyn, int n_wg,
                              hipStream_t s) {
  const dim3 grid(n_wg), block(64);
  if (st.kv8) {
    switch (group) {
    case 1: hipLaunchKernelGGL((k_step_valu<D, 1, true>), grid, block, 0, s, st, dyn); break;
    case 2: hipLaunchKernelGGL((k_step_valu<D, 2, true>), grid, block, 0, s, st, dyn); break;
    case 4: hipLaunchKernelGGL((k_step_valu<D, 4, true>), grid, block, 0, s, st, dyn); break;
    case 8: hipLaunchKernelGGL((k_step_valu<D, 8, true>), grid, block, 0, s, st, dyn); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (group) {
  case 1: hipLaunchKernelGGL((k_step_valu<D, 1, false>), grid, block, 0, s, st, dyn); break;
  case 2: hipLaunchKernelGGL((k_step_valu<D, 2, false>), grid, block, 0, s, st, dyn); break;
  case 4: hipLaunchKernelGGL((k_step_valu<D, 4, false>), grid, block, 0, s, st, dyn); break;
  case 8: hipLaunchKernelGGL((k_step_valu<D, 8, false>), grid, block, 0, s, st, dyn); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template <int D>
hipError_t step_mfma_dispatch(int group, const DecodeStatic &st, const DecodeDyn *dyn, int n_wg,
                              hipStream_t s) {
  constexpr int W = kMfmaWaves;
  const dim3 grid(n_wg), block(64 * W);
  if (st.kv8) {
    switch (group) {
    case 1: hipLaunchKernelGGL((k_step_mfma8<D, 1>), grid, block, 0, s, st, dyn); break;
    case 2: hipLaunchKernelGGL((k_step_mfma8<D, 2>), grid, block, 0, s, st, dyn); break;
    case 4: hipLaunchKernelGGL((k_step_mfma8<D, 4>), grid, block, 0, s, st, dyn); break;
    case 8: hipLaunchKernelGGL((k_step_mfma8<D, 8>), grid, block, 0, s, st, dyn); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (group) {
  case 1: hipLaunchKernelGGL((k_step_mfma<D, 1, W>), grid, block, 0, s, st, dyn); break;
  case 2: hipLaunchKernelGGL((k_step_mfma<D, 2, W>), grid, block, 0, s, st, dyn); break;
  case 4: hipLaunchKernelGGL((k_step_mfma<D, 4, W>), grid, block, 0, s, st, dyn); break;
  case 8: hipLaunchKernelGGL((k_step_mfma<D, 8, W>), grid, block, 0, s, st, dyn); break;
  default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
} // namespace

hipError_t launch_step_valu(int d, int group, const DecodeStatic &st, const DecodeDyn *dyn,
                            int n_wg, hipStream_t s) {
  if (n_wg <= 0) return hipErrorInvalidValue;
  return d == 128 ? step_valu_dispatch<128>(group, st, dyn, n_wg, s)
                  : step_valu_dispatch<64>(group, st, dyn, n_wg, s);
}

hipError_t launch_step_mfma(int d, int group, const DecodeStatic &st, const DecodeDyn *dyn,
                            int n_wg, hipStream_t s) {
  if (n_wg <= 0) return hipErrorInvalidValue;
  return d == 128 ? step_mfma_dispatch<128>(group, st, dyn, n_wg, s)
                  : step_mfma_dispatch<64>(group, st, dyn, n_wg, s);
}

hipError_t launch_step_merge(int d, int batch, const StepMergeArgs &a, bool kv8, hipStream_t s) {
  const dim3 grid(a.st.group, a.st.hkv, batch), block(64 * kMergeWaves);
  if (kv8) {
    if (d == 128)
      hipLaunchKernelGGL(k_step_merge8<128>, grid, block, 0, s, a);
    else
      hipLaunchKernelGGL(k_step_merge8<64>, grid, block, 0, s, a);
  } else if (d == 128)
    hipLaunchKernelGGL(k_step_merge<128>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_step_merge<64>, grid, block, 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Split partials of the allocation-free decode entry point: m [slots][kRows],
// l [slots][kRows], acc [slots][kRows][128] (64-channel heads use the first
// half of each acc slot's pitch-D rows), in a device array that every GPU the
// library runs on holds until the process ends.  Host code never uses the
// array's name as an address: the device address comes from
// hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) float scratch[kStaticSlots * kRows * (2 + 128)];

hipError_t static_partials(StaticPartials *out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  float *base = static_cast<float *>(addr[dev]);
  out->m = base;
  out->l = base + (int64_t)kStaticSlots * kRows;
  out->acc = base + 2 * (int64_t)kStaticSlots * kRows;
  out->slots = kStaticSlots;
  return hipSuccess;
}

} // namespace sq
