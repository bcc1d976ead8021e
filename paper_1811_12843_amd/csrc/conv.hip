// Convolutions of the DCGAN-style networks as implicit GEMMs on CDNA4 matrix
// cores (v_mfma_f32_16x16x4f32), and the fixed-order reductions around them:
// split-K weight-gradient sums with the Adam step, batch norm with batch
// statistics, and the logits of the 1-wide output layer.
//
// The convolution kernel never materialises an im2col matrix.  A workgroup
// (4 wave64) owns a 64 x 64 output tile (64 x 16 for outputs at most 16
// wide); K advances in 32-deep slices staged
// through a double-buffered LDS ring, the next slice's global loads in
// registers while the current one feeds the MFMAs.  Every operand element
// comes from a position map plus a tap shift (ConvProb, lipz_internal.h);
// taps that fall outside the image are loads at an offset past the
// operand's extent, which the buffer unit answers with 0 (the zero padding),
// so no load branches on the image border.
//
// Stride-2 transposed convolutions (the generator) and the input gradients
// of stride-2 convolutions (the discriminator) are split into their four
// output phases (sub-pixel decomposition): output (2y + r, 2x + q) only ever
// meets the 2 x 2 kernel taps of parity (r, q), so each phase is a dense
// 4-tap convolution and no zero-inserted input is multiplied.
//
// MFMA 16x16x4 f32 operand layout (wave64): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator register r of lane l is
// D[4 (l / 16) + r][l % 16].
#include <hip/hip_ext.h>

#include "lipz_internal.h"

namespace lipz {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

namespace {

constexpr int NT = 256;
constexpr int TM = 64, TK = 32;           // tile rows, K slice (tile columns: ConvProb::tn)
constexpr int SK = TK + 4;                // row stride of [row][k] LDS tiles
constexpr int SM = TM + 4;                // row stride of [k][m] tiles
constexpr int TILE_FLOATS = (TM * SK > TK * SM) ? TM * SK : TK * SM;
// A byte offset past every operand extent the host accepts: such a buffer
// load returns 0.
constexpr uint32_t OOB = 0x7FFFFFF0u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const float* p, uint32_t bytes) {
  // dword 3 = 0x00020000: raw 32-bit data format on gfx9-family parts
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 ld4(__amdgpu_buffer_rsrc_t r, uint32_t off_bytes) {
  const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off_bytes, 0, 0);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                     __uint_as_float(v[3]));
}
__device__ __forceinline__ float ld1(__amdgpu_buffer_rsrc_t r, uint32_t off_bytes) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)off_bytes, 0, 0));
}

// Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous range of logical tiles so neighbouring tiles share its L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, i = b >> 3;
  return x * q + (x < r ? x : r) + i;
}

struct Pos {
  int img, y, x;
};
__device__ __forceinline__ Pos grid_pos(int p, int gh, int gw) {
  return {p >> (gh + gw), (p >> gw) & ((1 << gh) - 1), p & ((1 << gw) - 1)};
}

// Tap t -> (row shift, column shift) of the gathered operand, and its
// weight-tap index kh * kw_full + kw.
struct Tap {
  int dy, dx, wt;
};
__device__ __forceinline__ Tap tap_of(const ConvProb& P, int t) {
  const int a = t >> P.tw_log, b = t & ((1 << P.tw_log) - 1);
  return {a * P.tys + P.ty0, b * P.tys + P.tx0, (a * P.khs + P.kh0) * P.kw_full + (b * P.khs + P.kw0)};
}

// k index of the tap-expanded operand -> (tap, channel).
__device__ __forceinline__ void split_k(const ConvProb& P, int k, int& t, int& c) {
  if (P.cs_log >= 0) {
    t = k >> P.cs_log;
    c = k & (P.cs - 1);
  } else if (P.taps <= 1) {
    t = 0;
    c = k;
  } else {
    t = k / P.cs;
    c = k - t * P.cs;
  }
}

// Byte offset of channel c of S at grid position q shifted by tap d, or OOB.
__device__ __forceinline__ uint32_t src_off(const ConvProb& P, Pos q, Tap d, int c) {
  const int sy = q.y * P.smap.sy + d.dy;
  const int sx = q.x * P.smap.sx + d.dx;
  if ((unsigned)sy >= (1u << P.smap.h_log) || (unsigned)sx >= (1u << P.smap.w_log)) return OOB;
  const int pos = (((q.img << P.smap.h_log) + sy) << P.smap.w_log) + sx;
  return (uint32_t)(pos * P.smap.ld + c) * 4u;
}

// Element offset (floats) of grid position q under a position map.
__device__ __forceinline__ int map_off(const PosMap& m, Pos q) {
  const int y = q.y * m.sy + m.y0, x = q.x * m.sx + m.x0;
  return ((((q.img << m.h_log) + y) << m.w_log) + x) * m.ld;
}

// ---------------------------------------------------------------------------
// Slice loads.  Thread tid loads two float4 groups of A and two of B per
// slice; the group -> (row, k) assignment matches the LDS layout written by
// store_slice.
//
//   CONV_FWD A [row][k]:  rows tid / 8 and 32 + tid / 8, k 4 (tid % 8)
//   CONV_WG  A [k][m]:    k tid / 16 and 16 + tid / 16, m 4 (tid % 16)
//   B [k][n] (BT 0):      k tid / 16 and 16 + tid / 16, n 4 (tid % 16)
//   B [n][k] (BT 1):      n tid / 8 and 32 + tid / 8, k 4 (tid % 8)
// ---------------------------------------------------------------------------
struct Ctx {
  __amdgpu_buffer_rsrc_t rs, rw, rp;
  Pos rowpos[2];  // FWD: grid positions of this thread's two A rows
  bool rowok[2];
  int mt[4], mc[4];   // WG: (tap, channel) of this thread's 4 A columns
  Tap mtap[4];
  int mkind[4];       // WG: 0 gathered, 1 ones row, 2 zero
};

template <int MODE, int GEN>
__device__ __forceinline__ void setup_ctx(const ConvProb& P, int m0, Ctx& X) {
  const int tid = threadIdx.x;
  X.rs = rsrc(P.S, P.s_bytes);
  if (MODE == CONV_FWD) {
    X.rw = rsrc(P.W, P.w_bytes);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int p = m0 + 32 * h + (tid >> 3);
      X.rowok[h] = p < P.M;
      X.rowpos[h] = grid_pos(p < P.M ? p : 0, P.gh_log, P.gw_log);
    }
  } else {
    X.rp = rsrc(P.P, P.p_bytes);
    const int mq = m0 + ((tid & 15) << 2);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = mq + e;
      int t = 0, c = 0;
      if (m < P.taps * P.cs) {
        split_k(P, m, t, c);
        X.mkind[e] = 0;
      } else {
        X.mkind[e] = (m == P.ones_row) ? 1 : 2;
      }
      X.mt[e] = t;
      X.mc[e] = c;
      X.mtap[e] = tap_of(P, t);
    }
  }
}

// Wave layout of a TM x TN_ tile.  TN_ = 64: 2 x 2 waves of 32 x 32 (2 x 2
// MFMA tiles each); TN_ = 16 (outputs at most 16 wide, such as 3 image
// channels): 4 waves of 16 x 16 (one MFMA tile each).
template <int TN_>
struct TW {
  static constexpr int TI = TN_ == 64 ? 2 : 1;  // MFMA tiles along m per wave
  static constexpr int TJ = TN_ == 64 ? 2 : 1;  // MFMA tiles along n per wave
  static constexpr int SN = TN_ + 4;            // row stride of [k][n] B tiles
  __device__ static int wm(int wave) { return TN_ == 64 ? (wave >> 1) * 32 : wave * 16; }
  __device__ static int wn(int wave) { return TN_ == 64 ? (wave & 1) * 32 : 0; }
};

// B group h of thread tid: (k row, first n) of a [k][n] slice, or (n row,
// first k) of an [n][k] slice; false when the thread has no such group
// (a 32 x 16 slice is 128 float4).
template <int TN_>
__device__ __forceinline__ bool b_kn(int h, int tid, int& kk, int& nq) {
  if (TN_ == 64) {
    kk = 16 * h + (tid >> 4);
    nq = (tid & 15) << 2;
    return true;
  }
  kk = tid >> 2;
  nq = (tid & 3) << 2;
  return h == 0 && tid < 128;
}
template <int TN_>
__device__ __forceinline__ bool b_nk(int h, int tid, int& nn, int& kq) {
  if (TN_ == 64) {
    nn = 32 * h + (tid >> 3);
    kq = (tid & 7) << 2;
    return true;
  }
  nn = tid >> 3;
  kq = (tid & 7) << 2;
  return h == 0 && tid < 128;
}

template <int MODE, int BT, int GEN, int TN_>
__device__ __forceinline__ void load_slice(const ConvProb& P, const Ctx& X, int n0, int k0, int kend,
                                           float4 (&ra)[2], float4 (&rb)[2]) {
  const int tid = threadIdx.x;
  if (MODE == CONV_FWD) {
    // A: gathered rows of the source; the 4 k of a group share one tap
    // unless the element-wise path is taken
    const int k = k0 + ((tid & 7) << 2);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (!GEN) {
        uint32_t off = OOB;
        if (X.rowok[h] && k < kend) {
          int t, c;
          split_k(P, k, t, c);
          off = src_off(P, X.rowpos[h], tap_of(P, t), c);
        }
        ra[h] = ld4(X.rs, off);
      } else {
        float e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t off = OOB;
          if (X.rowok[h] && k + e < kend) {
            int t, c;
            split_k(P, k + e, t, c);
            off = src_off(P, X.rowpos[h], tap_of(P, t), c);
          }
          e4[e] = ld1(X.rs, off);
        }
        ra[h] = make_float4(e4[0], e4[1], e4[2], e4[3]);
      }
    }
    // B: weights
    const int wtap = P.cs * P.N;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      rb[h] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (BT == 0) {
        int kr, nq;
        if (!b_kn<TN_>(h, tid, kr, nq)) continue;
        const int kk = k0 + kr, n = n0 + nq;
        int t = 0, c = 0;
        if (kk < kend) split_k(P, kk, t, c);
        const int base = tap_of(P, t).wt * wtap + c * P.wsc;
        if (!GEN) {
          const uint32_t off = (kk < kend && n < P.N) ? (uint32_t)(base + n) * 4u : OOB;
          rb[h] = ld4(X.rw, off);
        } else {
          float e4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int nn = n + e;
            const int no = P.n_inner ? (nn / P.n_inner) * P.n_tap_stride + (nn % P.n_inner) * P.wsn : nn * P.wsn;
            e4[e] = ld1(X.rw, (kk < kend && nn < P.N) ? (uint32_t)(base + no) * 4u : OOB);
          }
          rb[h] = make_float4(e4[0], e4[1], e4[2], e4[3]);
        }
      } else {
        int nr, kr;
        if (!b_nk<TN_>(h, tid, nr, kr)) continue;
        const int n = n0 + nr, kq = k0 + kr;
        if (!GEN) {
          uint32_t off = OOB;
          if (kq < kend && n < P.N) {
            int t, c;
            split_k(P, kq, t, c);
            off = (uint32_t)(tap_of(P, t).wt * wtap + c + n * P.wsn) * 4u;
          }
          rb[h] = ld4(X.rw, off);
        } else {
          float e4[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            uint32_t off = OOB;
            if (kq + e < kend && n < P.N) {
              int t, c;
              split_k(P, kq + e, t, c);
              off = (uint32_t)(tap_of(P, t).wt * wtap + c + n * P.wsn) * 4u;
            }
            e4[e] = ld1(X.rw, off);
          }
          rb[h] = make_float4(e4[0], e4[1], e4[2], e4[3]);
        }
      }
    }
  } else {
    // A [k = position][m = (tap, channel)]
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int p = k0 + 16 * h + (tid >> 4);
      const bool pok = p < kend;
      const Pos q = grid_pos(pok ? p : 0, P.gh_log, P.gw_log);
      if (!GEN) {
        // the 4 columns of a group share one tap (cs % 4 == 0)
        uint32_t off = OOB;
        if (pok && X.mkind[0] == 0) off = src_off(P, q, X.mtap[0], X.mc[0]);
        float4 v = ld4(X.rs, off);
        if (X.mkind[0] == 1) v = pok ? make_float4(1.f, 0.f, 0.f, 0.f) : make_float4(0.f, 0.f, 0.f, 0.f);
        ra[h] = v;
      } else {
        float e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t off = OOB;
          if (pok && X.mkind[e] == 0) off = src_off(P, q, X.mtap[e], X.mc[e]);
          const float v = ld1(X.rs, off);
          e4[e] = X.mkind[e] == 1 ? (pok ? 1.f : 0.f) : v;
        }
        ra[h] = make_float4(e4[0], e4[1], e4[2], e4[3]);
      }
    }
    // B [k = position][n]
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      rb[h] = make_float4(0.f, 0.f, 0.f, 0.f);
      int kr, nq;
      if (!b_kn<TN_>(h, tid, kr, nq)) continue;
      const int p = k0 + kr, n = n0 + nq;
      const bool pok = p < kend;
      const int base = pok ? map_off(P.pmap, grid_pos(p, P.gh_log, P.gw_log)) : 0;
      if (!GEN) {
        rb[h] = ld4(X.rp, (pok && n < P.N) ? (uint32_t)(base + n) * 4u : OOB);
      } else {
        float e4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) e4[e] = ld1(X.rp, (pok && n + e < P.N) ? (uint32_t)(base + n + e) * 4u : OOB);
        rb[h] = make_float4(e4[0], e4[1], e4[2], e4[3]);
      }
    }
  }
}

template <int MODE, int BT, int TN_>
__device__ __forceinline__ void store_slice(const float4 (&ra)[2], const float4 (&rb)[2], float* as, float* bs) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    float* da = MODE == CONV_FWD ? as + (32 * h + (tid >> 3)) * SK + ((tid & 7) << 2)
                                 : as + (16 * h + (tid >> 4)) * SM + ((tid & 15) << 2);
    *reinterpret_cast<float4*>(da) = ra[h];
    if (MODE == CONV_FWD && BT == 1) {
      int nr, kr;
      if (b_nk<TN_>(h, tid, nr, kr)) *reinterpret_cast<float4*>(bs + nr * SK + kr) = rb[h];
    } else {
      int kr, nq;
      if (b_kn<TN_>(h, tid, kr, nq)) *reinterpret_cast<float4*>(bs + kr * TW<TN_>::SN + nq) = rb[h];
    }
  }
}

// MFMAs of one slice in LDS: two 16-deep k blocks; in block kb, sub-step u
// of lane group g = l / 16 uses k = 16 kb + 4 g + u for both operands.
template <int MODE, int BT, int TN_>
__device__ __forceinline__ void mma_slice(const float* as, const float* bs, v4f (&acc)[2][2]) {
  using W = TW<TN_>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = W::wm(wave), wn = W::wn(wave);
  const int li = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < TK / 16; ++kb) {
    const int kq = 16 * kb + 4 * lg;
    float a[W::TI][4], b[W::TJ][4];
#pragma unroll
    for (int i = 0; i < W::TI; ++i) {
      const int m = wm + 16 * i + li;
      if (MODE == CONV_FWD) {
        const float4 v = *reinterpret_cast<const float4*>(as + m * SK + kq);
        a[i][0] = v.x; a[i][1] = v.y; a[i][2] = v.z; a[i][3] = v.w;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) a[i][u] = as[(kq + u) * SM + m];
      }
    }
#pragma unroll
    for (int j = 0; j < W::TJ; ++j) {
      const int n = wn + 16 * j + li;
      if (MODE == CONV_FWD && BT == 1) {
        const float4 v = *reinterpret_cast<const float4*>(bs + n * SK + kq);
        b[j][0] = v.x; b[j][1] = v.y; b[j][2] = v.z; b[j][3] = v.w;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) b[j][u] = bs[(kq + u) * W::SN + n];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < W::TI; ++i)
#pragma unroll
        for (int j = 0; j < W::TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][u], b[j][u], acc[i][j], 0, 0, 0);
  }
}

template <int MODE, int BT, int GEN, int TN_>
__device__ void conv_mainloop(const ConvProb& P, int m0, int n0, int kbeg, int kend, float* As, float* Bs,
                              v4f (&acc)[2][2]) {
  Ctx X;
  setup_ctx<MODE, GEN>(P, m0, X);
  float4 ra[2], rb[2];
  load_slice<MODE, BT, GEN, TN_>(P, X, n0, kbeg, kend, ra, rb);
  int it = 0;
  for (int k0 = kbeg; k0 < kend; k0 += TK, ++it) {
    float* as = As + (it & 1) * TILE_FLOATS;
    float* bs = Bs + (it & 1) * TILE_FLOATS;
    store_slice<MODE, BT, TN_>(ra, rb, as, bs);
    __syncthreads();
    if (k0 + TK < kend) load_slice<MODE, BT, GEN, TN_>(P, X, n0, k0 + TK, kend, ra, rb);
    mma_slice<MODE, BT, TN_>(as, bs, acc);
  }
}

template <int TN_>
__device__ __forceinline__ void conv_epilogue(const ConvProb& P, const v4f (&acc)[2][2], int m0, int n0, int split,
                                              float slope) {
  using W = TW<TN_>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = W::wm(wave), wn = W::wn(wave);
  const int li = lane & 15, lg = lane >> 4;
  LIPZ_GLOBAL float* gC = as_global(P.C);
  if (P.mode == CONV_WG) {
    gC += (int64_t)split * P.split_stride;
    // column part of the output offset, once per column
    int coff[W::TJ];
#pragma unroll
    for (int j = 0; j < W::TJ; ++j) {
      const int n = n0 + wn + 16 * j + li;
      coff[j] = n >= P.N ? -1 : (P.n_inner ? (n / P.n_inner) * P.n_tap_stride + n % P.n_inner : n);
    }
#pragma unroll
    for (int i = 0; i < W::TI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + 16 * i + 4 * lg + r;
        int crow = -1;
        if (m < P.taps * P.cs) {
          int t, c;
          split_k(P, m, t, c);
          crow = tap_of(P, t).wt * P.cs + c;
        } else if (m == P.ones_row) {
          crow = P.brow;
        }
        if (crow < 0 || m >= P.M) continue;
#pragma unroll
        for (int j = 0; j < W::TJ; ++j)
          if (coff[j] >= 0) gC[(int64_t)crow * P.ldc + coff[j]] = acc[i][j][r];
      }
    return;
  }
  float bias[2] = {0.f, 0.f};
  if (P.epi == EPI_BIAS_ACT && P.bias) {
#pragma unroll
    for (int j = 0; j < W::TJ; ++j) {
      const int n = n0 + wn + 16 * j + li;
      bias[j] = n < P.N ? as_global(P.bias)[n] : 0.f;
    }
  }
  const LIPZ_GLOBAL float* gAux = as_global(P.aux);
#pragma unroll
  for (int i = 0; i < W::TI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = m0 + wm + 16 * i + 4 * lg + r;
      if (p >= P.M) continue;
      const int base = map_off(P.omap, grid_pos(p, P.gh_log, P.gw_log));
#pragma unroll
      for (int j = 0; j < W::TJ; ++j) {
        const int n = n0 + wn + 16 * j + li;
        if (n >= P.N) continue;
        const int64_t o = (int64_t)base + n;
        float v = acc[i][j][r];
        if (P.epi == EPI_BIAS_ACT) v = act_fwd(P.act, v + bias[j], slope);
        else if (P.epi == EPI_DACT) v *= act_deriv_from_out(P.act, gAux[o], slope);
        gC[o] = v;
      }
    }
}

template <int TN_>
__device__ __forceinline__ void conv_tile(const ConvProb& P, int m0, int n0, int split, int kbeg, int kend, float slope,
                                          float* As, float* Bs) {
  v4f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  if (P.mode == CONV_FWD) {
    const bool bt = P.wsn != 1;
    if (P.gen) {
      if (bt) conv_mainloop<CONV_FWD, 1, 1, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
      else conv_mainloop<CONV_FWD, 0, 1, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
    } else {
      if (bt) conv_mainloop<CONV_FWD, 1, 0, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
      else conv_mainloop<CONV_FWD, 0, 0, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
    }
  } else {
    if (P.gen) conv_mainloop<CONV_WG, 0, 1, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
    else conv_mainloop<CONV_WG, 0, 0, TN_>(P, m0, n0, kbeg, kend, As, Bs, acc);
  }
  conv_epilogue<TN_>(P, acc, m0, n0, split, slope);
}

__global__ __launch_bounds__(NT, 2) void conv_kernel(const ConvProb* __restrict__ probs, ConvGroups grp,
                                                     float slope) {
  const int b = blockIdx.x;
  int gi = 0;
#pragma unroll
  for (int q = 1; q < GEMM_MAX_GROUPS; ++q)
    if (q < grp.n && b >= grp.first_block[q]) gi = q;
  // first_block is a multiple of 8, so (b - first_block) % 8 is still the XCD
  const int rel = xcd_remap(b - grp.first_block[gi], grp.blocks[gi]);
  if (rel >= grp.real_tiles[gi]) return;
  const int pi = grp.first_prob[gi] + rel / grp.tiles_per_prob[gi];
  const int lt = rel % grp.tiles_per_prob[gi];
  const ConvProb P = probs[pi];
  const int tiles_mn = P.tiles_m * P.tiles_n;
  const int split = lt / tiles_mn;
  const int rem = lt - split * tiles_mn;
  const int m0 = (rem / P.tiles_n) * TM;
  const int n0 = (rem % P.tiles_n) * P.tn;
  int kbeg = 0, kend = P.K;
  if (P.mode == CONV_WG) {
    kbeg = split * P.ksplit;
    kend = min(P.K, kbeg + P.ksplit);
  }
  __shared__ __align__(16) float As[2 * TILE_FLOATS];
  __shared__ __align__(16) float Bs[2 * TILE_FLOATS];
  if (P.tn == 16) conv_tile<16>(P, m0, n0, split, kbeg, kend, slope, As, Bs);
  else conv_tile<64>(P, m0, n0, split, kbeg, kend, slope, As, Bs);
}

// ---------------------------------------------------------------------------
// Split-K sums + Adam: thread e of descriptor d sums the splits of its
// gradient element in split order and takes the Adam step of the parameter.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void adam_at(float* p, float* m, float* v, float g, float lr, float bc1, float bc2,
                                        const AdamConsts& ac, float clip = 0.f) {
  const float mm = ac.beta1 * *m + ac.one_minus_beta1 * g;
  const float vv = ac.beta2 * *v + ac.one_minus_beta2 * g * g;
  *m = mm;
  *v = vv;
  float q = *p - lr * (mm / bc1) / (sqrtf(vv / bc2) + ac.eps);
  if (clip > 0.f) q = q > clip ? clip : (q < -clip ? -clip : q);  // keeps NaN
  *p = q;
}

// Grid (x, problem): the Adam bias corrections are computed once per thread,
// not per element.
__global__ void reduce_adam_kernel(const RedProb* __restrict__ probs, int step_local, AdamConsts ac) {
  const RedProb& R = probs[blockIdx.y];
  const int tt = *R.t + step_local + 1;
  const float bc1 = (float)(1.0 - pow((double)ac.beta1, (double)tt));
  const float bc2 = (float)(1.0 - pow((double)ac.beta2, (double)tt));
  const float lr = *R.lr;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < R.n; e += (int64_t)gridDim.x * blockDim.x) {
    float g = 0.f;
    for (int s = 0; s < R.splits; ++s) g += R.part[(int64_t)s * R.split_stride + e];
    adam_at(R.p + e, R.m + e, R.v + e, g, lr, bc1, bc2, ac, R.clip);
  }
}

// ---------------------------------------------------------------------------
// Batch norm.  Block b of an instance covers chunk b / groups (BN_CHUNK
// rows) and channel group b % groups (64 channels); thread (w, l) takes
// channel 64 g + l and rows w, w + 4, ... of the chunk.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_bn(const BnProb* probs, int n, int b) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].first_block <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Sum over the 4 row lanes of a channel, in a fixed order; every thread of
// the channel gets the result.
__device__ __forceinline__ float lanes4_sum(float x, float (*red)[64]) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  red[w][l] = x;
  __syncthreads();
  return (red[0][l] + red[1][l]) + (red[2][l] + red[3][l]);
}

__global__ __launch_bounds__(NT) void bn_chunk_stats_kernel(const BnProb* __restrict__ probs, int n_probs) {
  __shared__ float red[4][64];
  const BnProb& B = probs[find_bn(probs, n_probs, blockIdx.x)];
  const int groups = (B.ch + 63) / 64;
  const int lb = blockIdx.x - B.first_block;
  const int chunk = lb / groups, cg = lb % groups;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int ch = cg * 64 + l;
  const bool cok = ch < B.ch;
  const int64_t r0 = (int64_t)chunk * BN_CHUNK;
  const int nr = (int)min((int64_t)BN_CHUNK, B.rows - r0);
  float s = 0.f;
  for (int r = w; r < nr; r += 4) s += cok ? B.x[(r0 + r) * B.ch + ch] : 0.f;
  const float mean = lanes4_sum(s, red) / (float)nr;
  float q = 0.f;
  for (int r = w; r < nr; r += 4) {
    const float d = (cok ? B.x[(r0 + r) * B.ch + ch] : 0.f) - mean;
    q += d * d;
  }
  const float m2 = lanes4_sum(q, red);
  if (w == 0 && cok) {
    B.part[((int64_t)chunk * 2 + 0) * B.ch + ch] = mean;
    B.part[((int64_t)chunk * 2 + 1) * B.ch + ch] = m2;
  }
}

// One thread per (instance, channel): merge the chunks in order.
__global__ void bn_merge_stats_kernel(const BnProb* __restrict__ probs, int n_probs, int max_ch, float eps) {
  const int i = blockIdx.y;
  const int ch = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_probs || ch >= probs[i].ch || ch >= max_ch) return;
  const BnProb& B = probs[i];
  const int chunks = (int)((B.rows + BN_CHUNK - 1) / BN_CHUNK);
  double n_a = 0.0;
  float mean = 0.f, m2 = 0.f;
  for (int k = 0; k < chunks; ++k) {
    const float n_b = (float)min((int64_t)BN_CHUNK, B.rows - (int64_t)k * BN_CHUNK);
    const float mb = B.part[((int64_t)k * 2 + 0) * B.ch + ch];
    const float qb = B.part[((int64_t)k * 2 + 1) * B.ch + ch];
    const float n = (float)n_a + n_b;
    const float d = mb - mean;
    mean += d * (n_b / n);
    m2 += qb + d * d * ((float)n_a * n_b / n);
    n_a += n_b;
  }
  const float var = m2 / (float)B.rows;
  B.stats[ch] = mean;
  B.stats[B.ch + ch] = 1.f / sqrtf(var + eps);
}

// y = act(gamma (x - mean) rstd + beta), 4 channels per thread.
__global__ void bn_apply_kernel(const BnProb* __restrict__ probs, int n_probs, float slope) {
  const int i = blockIdx.y;
  if (i >= n_probs) return;
  const BnProb& B = probs[i];
  const int64_t n4 = B.rows * B.ch / 4;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n4; q += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)((q * 4) % B.ch);
    const float4 x = reinterpret_cast<const float4*>(B.x)[q];
    float xv[4] = {x.x, x.y, x.z, x.w}, yv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float h = (xv[e] - B.stats[c + e]) * B.stats[B.ch + c + e];
      yv[e] = act_fwd(B.act, B.gamma[c + e] * h + B.gamma[B.ch + c + e], slope);
    }
    reinterpret_cast<float4*>(B.y)[q] = make_float4(yv[0], yv[1], yv[2], yv[3]);
  }
}

// Backward, stage 1: per chunk, sum of dy and of dy * xhat.
__global__ __launch_bounds__(NT) void bn_chunk_grad_kernel(const BnProb* __restrict__ probs, int n_probs) {
  __shared__ float red[4][64];
  const BnProb& B = probs[find_bn(probs, n_probs, blockIdx.x)];
  const int groups = (B.ch + 63) / 64;
  const int lb = blockIdx.x - B.first_block;
  const int chunk = lb / groups, cg = lb % groups;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int ch = cg * 64 + l;
  const bool cok = ch < B.ch;
  const int64_t r0 = (int64_t)chunk * BN_CHUNK;
  const int nr = (int)min((int64_t)BN_CHUNK, B.rows - r0);
  const float mean = cok ? B.stats[ch] : 0.f, rstd = cok ? B.stats[B.ch + ch] : 0.f;
  float s = 0.f, sx = 0.f;
  for (int r = w; r < nr; r += 4) {
    if (!cok) break;
    const int64_t o = (r0 + r) * B.ch + ch;
    const float dy = B.y[o];
    s += dy;
    sx += dy * ((B.x[o] - mean) * rstd);
  }
  s = lanes4_sum(s, red);
  sx = lanes4_sum(sx, red);
  if (w == 0 && cok) {
    B.part[((int64_t)chunk * 2 + 0) * B.ch + ch] = s;
    B.part[((int64_t)chunk * 2 + 1) * B.ch + ch] = sx;
  }
}

// Stage 2: per channel, the sums in chunk order -> coefficients of dx
// (gamma rstd, dbeta / R, dgamma / R, with the gamma before this step),
// then the Adam steps of gamma and beta.
__global__ void bn_merge_grad_kernel(const BnProb* __restrict__ probs, int n_probs, int max_ch, int step_local,
                                     AdamConsts ac) {
  const int i = blockIdx.y;
  const int ch = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_probs || ch >= probs[i].ch || ch >= max_ch) return;
  const BnProb& B = probs[i];
  const int chunks = (int)((B.rows + BN_CHUNK - 1) / BN_CHUNK);
  float db = 0.f, dg = 0.f;
  for (int k = 0; k < chunks; ++k) {
    db += B.part[((int64_t)k * 2 + 0) * B.ch + ch];
    dg += B.part[((int64_t)k * 2 + 1) * B.ch + ch];
  }
  const float R = (float)B.rows;
  B.stats[2 * B.ch + ch] = B.gamma[ch] * B.stats[B.ch + ch];
  B.stats[3 * B.ch + ch] = db / R;
  B.stats[4 * B.ch + ch] = dg / R;
  const int tt = *B.t + step_local + 1;
  const float bc1 = (float)(1.0 - pow((double)ac.beta1, (double)tt));
  const float bc2 = (float)(1.0 - pow((double)ac.beta2, (double)tt));
  const float lr = *B.lr;
  adam_at(B.gamma + ch, B.gm + ch, B.gv + ch, dg, lr, bc1, bc2, ac);
  adam_at(B.gamma + B.ch + ch, B.gm + B.ch + ch, B.gv + B.ch + ch, db, lr, bc1, bc2, ac);
}

// Stage 3: dx = gamma rstd (dy - dbeta / R - xhat dgamma / R), in place.
__global__ void bn_apply_grad_kernel(const BnProb* __restrict__ probs, int n_probs) {
  const int i = blockIdx.y;
  if (i >= n_probs) return;
  const BnProb& B = probs[i];
  const int64_t n4 = B.rows * B.ch / 4;
  const float* st = B.stats;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n4; q += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)((q * 4) % B.ch);
    const float4 x = reinterpret_cast<const float4*>(B.x)[q];
    const float4 d = reinterpret_cast<const float4*>(B.y)[q];
    const float xv[4] = {x.x, x.y, x.z, x.w}, dv[4] = {d.x, d.y, d.z, d.w};
    float o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int cc = c + e;
      const float h = (xv[e] - st[cc]) * st[B.ch + cc];
      o[e] = st[2 * B.ch + cc] * (dv[e] - st[3 * B.ch + cc] - h * st[4 * B.ch + cc]);
    }
    reinterpret_cast<float4*>(B.y)[q] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// ---------------------------------------------------------------------------
// Logits of a 1-wide dense layer: block r computes row r's dot product
// (lane-strided float4 partial sums, then a fixed-order tree).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_dot(const DotProb* probs, int n, int r) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].first_row <= r) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(NT) void dot_rows_kernel(const DotProb* __restrict__ probs, int n_probs) {
  __shared__ float red[NT / 64];
  const DotProb& D = probs[find_dot(probs, n_probs, blockIdx.x)];
  const int r = blockIdx.x - D.first_row;
  const float* x = D.x + (int64_t)r * D.H;
  float s = 0.f;
  if ((D.H & 3) == 0 && ((((uintptr_t)x) | ((uintptr_t)D.w)) & 15) == 0) {
    for (int k = threadIdx.x * 4; k < D.H; k += NT * 4) {
      const float4 a = *reinterpret_cast<const float4*>(x + k);
      const float4 b = *reinterpret_cast<const float4*>(D.w + k);
      s += (a.x * b.x + a.y * b.y) + (a.z * b.z + a.w * b.w);
    }
  } else {
    for (int k = threadIdx.x; k < D.H; k += NT) s += x[k] * D.w[k];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) D.out[(int64_t)r * D.ld_out] = ((red[0] + red[1]) + (red[2] + red[3])) + D.w[D.H];
}

// ---------------------------------------------------------------------------
// DCGAN initialisation.
// ---------------------------------------------------------------------------
__global__ void init_conv_params_kernel(float* p, int64_t stride, int64_t P, int C, ConvInitLayout L, uint2 key,
                                        uint32_t tag) {
  const int64_t total = (int64_t)C * P;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i / P);
    const int64_t e = i - (int64_t)c * P;
    int kind = 0;  // 0: zero, 1: weight, 2: gamma
    for (int l = 0; l < L.n; ++l) {
      if (e >= L.off_w[l] && e < L.off_w[l] + L.n_w[l]) kind = 1;
      if (L.n_g[l] > 0 && e >= L.off_g[l] && e < L.off_g[l] + L.n_g[l]) kind = 2;
    }
    float v = 0.f;
    if (kind) {
      const uint4 w = stream_block(key, (uint32_t)(e >> 2), (uint32_t)c, 0, 0, tag);
      const double n = normal_of(w, (int)(e & 3));
      v = (float)(kind == 1 ? 0.02 * n : 1.0 + 0.02 * n);
    }
    p[(int64_t)c * stride + e] = v;
  }
}

// ---------------------------------------------------------------------------
// Patches and their inverse gather (ColProb, lipz_internal.h).  Grid (x,
// descriptor).  im2col: one thread per (position, tap) copies its ch
// channels; col2im: one thread per output element.
// ---------------------------------------------------------------------------
__global__ void im2col_kernel(const ColProb* __restrict__ probs) {
  const ColProb& Q = probs[blockIdx.y];
  const int g = Q.h_log - 1;  // grid side log2
  const int S = 1 << Q.h_log;
  const int64_t n = ((int64_t)Q.n_img << (2 * g)) * 16;  // (position, tap) pairs
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int t = (int)(i & 15);
    const int64_t p = i >> 4;
    const int img = (int)(p >> (2 * g)), y = (int)((p >> g) & ((1 << g) - 1)), x = (int)(p & ((1 << g) - 1));
    const int sy = 2 * y - 1 + (t >> 2), sx = 2 * x - 1 + (t & 3);
    const bool in = sy >= 0 && sy < S && sx >= 0 && sx < S;
    const float* src = Q.src + (((int64_t)img * S + (in ? sy : 0)) * S + (in ? sx : 0)) * Q.ch;
    float* dst = Q.dst + i * Q.ch;
    for (int c = 0; c < Q.ch; ++c) dst[c] = in ? src[c] : 0.f;
  }
}

__global__ void col2im_kernel(const ColProb* __restrict__ probs, float slope) {
  const ColProb& Q = probs[blockIdx.y];
  const int S = 1 << Q.h_log, Gs = S >> 1;
  const int64_t n = ((int64_t)Q.n_img << (2 * Q.h_log)) * Q.ch;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(e % Q.ch);
    const int64_t pix = e / Q.ch;
    const int X = (int)(pix & (S - 1)), Y = (int)((pix >> Q.h_log) & (S - 1));
    const int img = (int)(pix >> (2 * Q.h_log));
    float s = 0.f;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int kh = ((Y + 1) & 1) + 2 * a;
      const int iy = (Y + 1 - kh) >> 1;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int kw = ((X + 1) & 1) + 2 * b;
        const int ix = (X + 1 - kw) >> 1;
        if (iy >= 0 && iy < Gs && ix >= 0 && ix < Gs)
          s += Q.src[(((int64_t)img * Gs + iy) * Gs + ix) * (16 * Q.ch) + (kh * 4 + kw) * Q.ch + c];
      }
    }
    if (Q.epi == EPI_BIAS_ACT) s = act_fwd(Q.act, s + (Q.bias ? Q.bias[c] : 0.f), slope);
    else if (Q.epi == EPI_DACT) s *= act_deriv_from_out(Q.act, Q.aux[e], slope);
    Q.dst[e] = s;
  }
}

int blocks_for(int64_t n, int cap = 16384) {
  const int64_t b = (n + NT - 1) / NT;
  return (int)(b < 1 ? 1 : (b > cap ? cap : b));
}

}  // namespace

hipError_t launch_conv_grouped(const ConvProb* d_probs, const ConvGroups& grp, int total_blocks, float slope,
                               hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (grp.n <= 0 || total_blocks <= 0) return hipSuccess;
  hipExtLaunchKernelGGL(conv_kernel, dim3(total_blocks), dim3(NT), 0, s, ev_start, ev_stop, 0, d_probs, grp, slope);
  return hipGetLastError();
}

hipError_t launch_reduce_adam(const RedProb* d_probs, int n_probs, int64_t max_n, int step_local, AdamConsts ac,
                              hipStream_t s) {
  if (n_probs <= 0 || max_n <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_adam_kernel, dim3(blocks_for(max_n, 2048), n_probs), dim3(NT), 0, s, d_probs, step_local,
                     ac);
  return hipGetLastError();
}

hipError_t launch_bn_stats(const BnProb* d_probs, int n_probs, int total_blocks, float eps, hipStream_t s) {
  if (n_probs <= 0) return hipSuccess;
  hipLaunchKernelGGL(bn_chunk_stats_kernel, dim3(total_blocks), dim3(NT), 0, s, d_probs, n_probs);
  hipLaunchKernelGGL(bn_merge_stats_kernel, dim3(4, n_probs), dim3(NT), 0, s, d_probs, n_probs, 4 * NT, eps);
  return hipGetLastError();
}

hipError_t launch_bn_apply(const BnProb* d_probs, int n_probs, int64_t max_elems, float slope, hipStream_t s) {
  if (n_probs <= 0) return hipSuccess;
  hipLaunchKernelGGL(bn_apply_kernel, dim3(blocks_for(max_elems / 4, 4096), n_probs), dim3(NT), 0, s, d_probs,
                     n_probs, slope);
  return hipGetLastError();
}

hipError_t launch_bn_backward(const BnProb* d_probs, int n_probs, int total_blocks, int64_t max_elems,
                              int step_local, AdamConsts ac, hipStream_t s) {
  if (n_probs <= 0) return hipSuccess;
  hipLaunchKernelGGL(bn_chunk_grad_kernel, dim3(total_blocks), dim3(NT), 0, s, d_probs, n_probs);
  hipLaunchKernelGGL(bn_merge_grad_kernel, dim3(4, n_probs), dim3(NT), 0, s, d_probs, n_probs, 4 * NT, step_local,
                     ac);
  hipLaunchKernelGGL(bn_apply_grad_kernel, dim3(blocks_for(max_elems / 4, 4096), n_probs), dim3(NT), 0, s, d_probs,
                     n_probs);
  return hipGetLastError();
}

hipError_t launch_dot_rows(const DotProb* d_probs, int n_probs, int total_rows, hipStream_t s) {
  if (n_probs <= 0 || total_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(dot_rows_kernel, dim3(total_rows), dim3(NT), 0, s, d_probs, n_probs);
  return hipGetLastError();
}

hipError_t launch_im2col(const ColProb* d_probs, int n_probs, int64_t max_pairs, hipStream_t s) {
  if (n_probs <= 0 || max_pairs <= 0) return hipSuccess;
  hipLaunchKernelGGL(im2col_kernel, dim3(blocks_for(max_pairs, 8192), n_probs), dim3(NT), 0, s, d_probs);
  return hipGetLastError();
}

hipError_t launch_col2im(const ColProb* d_probs, int n_probs, int64_t max_elems, float slope, hipStream_t s) {
  if (n_probs <= 0 || max_elems <= 0) return hipSuccess;
  hipLaunchKernelGGL(col2im_kernel, dim3(blocks_for(max_elems, 8192), n_probs), dim3(NT), 0, s, d_probs, slope);
  return hipGetLastError();
}

hipError_t launch_init_conv_params(float* p, int64_t stride, int64_t P, int C, const ConvInitLayout& L, uint2 key,
                                   uint32_t tag, hipStream_t s) {
  hipLaunchKernelGGL(init_conv_params_kernel, dim3(blocks_for((int64_t)C * P)), dim3(NT), 0, s, p, stride, P, C, L,
                     key, tag);
  return hipGetLastError();
}

}  // namespace lipz
