// Implicit-GEMM engine for convolution and linear layers on CDNA4 MFMA.
//
// Two precisions share one structure:
//   bf16 storage: operands are bf16, v_mfma_f32_16x16x32_bf16, fp32 accumulators;
//   fp32 storage: operands are fp32, widened to fp64 and multiplied with
//                 v_mfma_f64_16x16x4f64 (fp64 accumulators), so every output is
//                 the nearest fp32 of an (almost) exact dot product.
// A 256-thread workgroup (4 wave64s) owns a BM x BN output tile.  Operand
// tiles are staged through LDS in 16-byte chunks, double-buffered: the global
// loads of step k+1 are in flight while the MFMAs of step k run.
//
// Forward-type GEMM (k_conv_gemm): rows m = output pixels, columns n = output
// channels, reduction over (r, s, c) of the zero-padded input window.  The
// A tile is gathered straight from the NHWC input (implicit im2col); with a
// channel count that is a multiple of the 16-byte chunk, a reduction step
// covers one (r, s) tap and a run of channels, otherwise every element is
// gathered on its own ("flat" mode, used by 3-channel image inputs).
//
// Weight-gradient GEMM (k_wgrad): rows = output channels, columns = (r, s, c),
// reduction over the pixels of the micro-batch.  The pixel range is split
// over blockIdx.z; each split writes its partial tile to a workspace and a
// second kernel adds the splits in a fixed order into the fp32 gradient
// accumulator (deterministic, no atomics).
#include "xp_device.h"
#include <type_traits>
#include "xp_kernels.h"

#include <cstdio>
#include <cstdlib>

namespace xp {

template <typename T> struct MT;
template <> struct MT<bf16_t> {
  static constexpr int VEC = 8;     // elements per 16-byte chunk
  typedef f32x4_t acc_t;
  typedef float part_t;
  static XP_DEV int out_row(int lane, int q) { return 4 * (lane >> 4) + q; }
};
template <> struct MT<float> {
  static constexpr int VEC = 4;
  typedef f64x4_t acc_t;
  typedef double part_t;
  static XP_DEV int out_row(int lane, int q) { return (lane >> 4) + 4 * q; }
};

template <typename T>
XP_DEV T zero_elem() { return T(0); }

// pack VEC scalars (as raw bits) into a 16-byte chunk
template <typename T>
XP_DEV uint4 pack_chunk(const T* v);
template <>
XP_DEV uint4 pack_chunk<bf16_t>(const bf16_t* v) {
  uint4 r;
  r.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
  r.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
  r.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
  r.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
  return r;
}
template <>
XP_DEV uint4 pack_chunk<float>(const float* v) {
  uint4 r;
  r.x = __float_as_uint(v[0]);
  r.y = __float_as_uint(v[1]);
  r.z = __float_as_uint(v[2]);
  r.w = __float_as_uint(v[3]);
  return r;
}

// ============================================================================
// forward-type implicit GEMM
// ============================================================================
// KS sets the stage depth BK = KS x 32 (bf16: one v_mfma_f32_16x16x32_bf16 per
// 32) or KS x 16 (fp32 storage: four v_mfma_f64_16x16x4f64 per 16); deeper
// stages keep more bytes in flight per barrier.
// LDS row padding of the bf16 operand tiles, in elements
#ifndef XP_GEMM_LDS_PAD_BF16
#define XP_GEMM_LDS_PAD_BF16 16
#endif

// calls f(integral_constant<int, I>) for I = B .. E-1
template <int B, int E, typename F>
XP_DEV void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}


// bf16 epilogue from the fp32 result tile staged in LDS (ot, BM rows of
// OPITCH floats; every thread of the workgroup takes part): each thread
// finishes 8-column chunks of a row (bias, ReLU, mask, accumulate, round
// once) with 16-byte loads and stores, leaves the stored values in LDS, and
// the batch-norm column statistics of the tile are taken from there.
template <int BM, int BN, int NT, int OPITCH>
XP_DEV void conv_epilogue_bf16(const ConvArgs& a, float* ot, int tid, int m0, int n0, int tm, int M,
                               int row_tiles) {
  typedef bf16_t T;
  T* __restrict__ y = (T*)a.y;
  const T* __restrict__ mask = (const T*)a.mask;
  constexpr int CPRN = BN / 8;  // 8-column chunks per tile row
  static_assert(BN % 8 == 0, "chunked epilogue");
  // 16-byte global access needs 8-element aligned rows and base pointers
  const bool vy = (a.ldy % 8) == 0 && (reinterpret_cast<uintptr_t>(y) % 16) == 0;
  const bool vm = mask && (a.ldm % 8) == 0 && (reinterpret_cast<uintptr_t>(mask) % 16) == 0;
  // all loads of the thread's chunks are issued before its first store (a
  // load after a store waits for the store on this hardware); full chunks
  // take 16-byte accesses, a ragged last chunk (N not a multiple of 8) or
  // unaligned views an element loop
  typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
  constexpr int NCH = (BM * CPRN + NT - 1) / NT;  // chunks per thread
  int c_ne[NCH];
  u32x4_t c_mask[NCH], c_old[NCH];
  f32x4_t c_b0[NCH], c_b1[NCH];
  const bool vb = a.bias && (reinterpret_cast<uintptr_t>(a.bias + n0) % 16) == 0;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int c = k * NT + tid;
    const int row = c / CPRN, cc = c - row * CPRN;
    const int m = m0 + row, nb = n0 + cc * 8;
    const bool live = ((BM * CPRN) % NT == 0 || c < BM * CPRN) && m < M && nb < a.N;
    const int ne = live ? (a.N - nb < 8 ? a.N - nb : 8) : 0;  // valid columns in this chunk
    c_ne[k] = ne;
    c_mask[k] = c_old[k] = (u32x4_t){0u, 0u, 0u, 0u};
    c_b0[k] = c_b1[k] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    if (ne == 8) {
      if (vb) {
        c_b0[k] = *reinterpret_cast<const f32x4_t*>(a.bias + nb);
        c_b1[k] = *reinterpret_cast<const f32x4_t*>(a.bias + nb + 4);
      }
      if (vm) c_mask[k] = *reinterpret_cast<const u32x4_t*>(mask + (size_t)m * a.ldm + nb);
      if (a.accumulate && vy) c_old[k] = *reinterpret_cast<const u32x4_t*>(y + (size_t)m * a.ldy + nb);
    }
    if (ne > 0 && (ne < 8 || (a.bias && !vb) || (mask && !vm) || (a.accumulate && !vy))) {
      float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      uint16_t mv[8] = {0, 0, 0, 0, 0, 0, 0, 0}, ov[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      for (int e = 0; e < ne; ++e) {
        if (a.bias) bv[e] = a.bias[nb + e];
        if (mask) mv[e] = mask[(size_t)m * a.ldm + nb + e];
        if (a.accumulate) ov[e] = y[(size_t)m * a.ldy + nb + e];
      }
      c_b0[k] = (f32x4_t){bv[0], bv[1], bv[2], bv[3]};
      c_b1[k] = (f32x4_t){bv[4], bv[5], bv[6], bv[7]};
      c_mask[k] = *reinterpret_cast<const u32x4_t*>(mv);
      c_old[k] = *reinterpret_cast<const u32x4_t*>(ov);
    }
  }
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int c = k * NT + tid;
    if ((BM * CPRN) % NT != 0 && c >= BM * CPRN) break;
    const int row = c / CPRN, cc = c - row * CPRN;
    const int ne = c_ne[k];
    float* o = &ot[row * OPITCH + cc * 8];
    if (ne > 0) {
      const f32x4_t lo = *reinterpret_cast<const f32x4_t*>(o);
      const f32x4_t hi = *reinterpret_cast<const f32x4_t*>(o + 4);
      float f[8];
      if (!a.accumulate) {
        // one rounding to fp32 of acc + bias equals the rounding of their
        // exact double sum (53 >= 2 * 24 + 2), and ReLU and the mask commute
        // with rounding, so fp32 arithmetic stores the same values
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          f[e] = lo[e] + c_b0[k][e];
          f[e + 4] = hi[e] + c_b1[k][e];
        }
      } else {
        // y + result: added to the double value, rounded once
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          double v = (double)(e < 4 ? lo[e] : hi[e - 4]) + (double)(e < 4 ? c_b0[k][e] : c_b1[k][e - 4]);
          if (a.relu) v = v > 0.0 ? v : 0.0;
          const uint32_t mw = c_mask[k][e >> 1];
          if (mask && !(__uint_as_float((e & 1) ? (mw & 0xffff0000u) : (mw << 16)) > 0.0f)) v = 0.0;
          const uint32_t ow = c_old[k][e >> 1];
          v += (double)__uint_as_float((e & 1) ? (ow & 0xffff0000u) : (ow << 16));
          f[e] = (float)v;
        }
      }
      if (!a.accumulate) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (a.relu) f[e] = f[e] > 0.f ? f[e] : 0.f;
          const uint32_t mw = c_mask[k][e >> 1];
          if (mask && !(__uint_as_float((e & 1) ? (mw & 0xffff0000u) : (mw << 16)) > 0.0f)) f[e] = 0.f;
        }
      }
      u32x4_t pr;
#pragma unroll
      for (int q = 0; q < 4; ++q) pr[q] = f32x2_to_bf16x2(f[2 * q], f[2 * q + 1]);
      T* p = y + (size_t)(m0 + row) * a.ldy + n0 + cc * 8;
      if (vy && ne == 8) {
        *reinterpret_cast<u32x4_t*>(p) = pr;
      } else {
        for (int e = 0; e < ne; ++e) p[e] = (uint16_t)(pr[e >> 1] >> ((e & 1) * 16));
      }
      if (a.stat_part || a.bn_part) {
        f32x4_t s0, s1;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          s0[2 * q] = 2 * q < ne ? __uint_as_float(pr[q] << 16) : 0.f;
          s0[2 * q + 1] = 2 * q + 1 < ne ? __uint_as_float(pr[q] & 0xffff0000u) : 0.f;
          s1[2 * q] = 2 * q + 4 < ne ? __uint_as_float(pr[q + 2] << 16) : 0.f;
          s1[2 * q + 1] = 2 * q + 5 < ne ? __uint_as_float(pr[q + 2] & 0xffff0000u) : 0.f;
        }
        *reinterpret_cast<f32x4_t*>(o) = s0;
        *reinterpret_cast<f32x4_t*>(o + 4) = s1;
      }
    } else if (a.stat_part || a.bn_part) {
      *reinterpret_cast<f32x4_t*>(o) = (f32x4_t){0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<f32x4_t*>(o + 4) = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    }
  }
  if (a.stat_part || a.bn_part) {
    // per column, over the tile's rows, the sums of the stored values and of
    // their squares (batch-norm statistics), or, for a stored gradient g of a
    // batch norm with input z (bn_part), the sums of g and of g (z - mean) rstd
    // (its backward partials; z read a row at a time, columns across
    // threads): RS row ranges per column, each with four interleaved fp64
    // sums, then a fixed-order sum of the ranges
    constexpr int RS = NT / BN > 0 ? NT / BN : 1;
    constexpr int RROWS = BM / RS;
    static_assert(BM % RS == 0 && RROWS % 4 == 0, "row ranges");
    __shared__ double sred[RS][2][BN];
    __syncthreads();
    if (tid < RS * BN) {
      const int col = tid % BN, part = tid / BN;
      const float* oc = ot + part * RROWS * OPITCH + col;
      double s0[4] = {0.0, 0.0, 0.0, 0.0}, s1[4] = {0.0, 0.0, 0.0, 0.0};
      if (!a.bn_part) {
#pragma unroll
        for (int r = 0; r < RROWS; ++r) {
          const double sv = (double)oc[r * OPITCH];
          s0[r & 3] += sv;
          s1[r & 3] += sv * sv;
        }
      } else {
        // the batch norm this column belongs to (selected with constant
        // indices: no dynamic indexing of the argument arrays)
        const int n = n0 + col, mr = m0 + part * RROWS;
        const bf16_t* zc = nullptr;
        const double *mp = nullptr, *rp = nullptr;
        int ldz = 0;
        bool sum_only = false;  // a bias (no z): the column sums of g alone
#pragma unroll
        for (int q = 0; q < CONV_BN_SEGS; ++q)
          if (q < a.bn_nseg && n >= a.bn_c0[q] && n < a.bn_c1[q]) {
            const int lc = n - a.bn_c0[q];
            sum_only = a.bn_z[q] == nullptr;
            zc = sum_only ? nullptr : (const bf16_t*)a.bn_z[q] + lc;
            ldz = a.ld_bnz[q];
            mp = sum_only ? nullptr : a.bn_mean[q] + lc;
            rp = sum_only ? nullptr : a.bn_rstd[q] + lc;
          }
        if (sum_only && n < a.N) {
#pragma unroll
          for (int r = 0; r < RROWS; ++r) s0[r & 3] += (double)oc[r * OPITCH];  // 0 past the last row
        } else if (zc && n < a.N) {
          const double mu = *mp, rs = *rp;
          // every load issued before the first use: rows past the last are
          // read at the last row (their g is 0)
          float zv[RROWS];
#pragma unroll
          for (int r = 0; r < RROWS; ++r) zv[r] = bf16_to_f32(zc[(size_t)min(mr + r, M - 1) * ldz]);
#pragma unroll
          for (int r = 0; r < RROWS; ++r) {
            const double g = (double)oc[r * OPITCH];  // 0 past the last row
            s0[r & 3] += g;
            s1[r & 3] += g * (((double)zv[r] - mu) * rs);
          }
        }
      }
      sred[part][0][col] = (s0[0] + s0[1]) + (s0[2] + s0[3]);
      sred[part][1][col] = (s1[0] + s1[1]) + (s1[2] + s1[3]);
    }
    __syncthreads();
    double* part_out = a.bn_part ? a.bn_part : a.stat_part;
    for (int col = tid; col < BN; col += NT) {
      const int n = n0 + col;
      if (n >= a.N) continue;
      double s0 = 0.0, s1 = 0.0;
#pragma unroll
      for (int q = 0; q < RS; ++q) {
        s0 += sred[q][0][col];
        s1 += sred[q][1][col];
      }
      part_out[((size_t)n * 2 + 0) * row_tiles + tm] = s0;
      part_out[((size_t)n * 2 + 1) * row_tiles + tm] = s1;
    }
  }
}

// GM selects the gather: 0 stride 1 (rows = input grid), 1 strided forward,
// 2 strided data gradient (see ConvArgs)
template <typename T, int BM, int BN, int WM, int WN, bool FLAT, int KS, int PF, int GM>
__global__ __launch_bounds__(WM * WN * 64) void k_conv_gemm(ConvArgs a) {
  constexpr int NT = WM * WN * 64;  // threads: one wave64 per wave tile
  using MTT = MT<T>;
  constexpr int VEC = MTT::VEC;
  constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
  // bf16 wave tiles that are multiples of 32 use v_mfma_f32_32x32x16_bf16,
  // which on gfx950 has twice the throughput of the 16x16x32 form, and step
  // through K in multiples of 16 (KS counts 16-deep slices); otherwise KS
  // counts 32-deep slices (bf16, 16x16x32) or 16-deep (fp32 storage, f64 MFMA)
  constexpr bool M32 = sizeof(T) == 2 && WTM % 32 == 0 && WTN % 32 == 0;
  constexpr int SUB = (sizeof(T) == 2 && !M32) ? 32 : 16;
  constexpr int BK = KS * SUB;
  constexpr int PITCH = BK + (sizeof(T) == 2 ? XP_GEMM_LDS_PAD_BF16 : 4);
  constexpr int CPR = BK / VEC;  // chunks per tile row per step
  constexpr int A_CH = BM * CPR, B_CH = BN * CPR;
  constexpr int A_PER = (A_CH + NT - 1) / NT, B_PER = (B_CH + NT - 1) / NT;
  static_assert(WM * WN >= 1 && WM * WN <= 8, "one to eight waves");
  static_assert(TM >= 1 && TN >= 1, "wave tile");
  // bf16: the epilogue stages the fp32 result tile in the same LDS, rows
  // padded so that the accumulator layouts write it without bank conflicts
  constexpr int OPITCH = BN + (M32 ? 8 : 4);
  constexpr int STAGE_BYTES = 2 * (BM + BN) * PITCH * (int)sizeof(T);
  constexpr int OUT_BYTES = sizeof(T) == 2 ? BM * OPITCH * 4 : 0;
  __shared__ __align__(16) unsigned char smem[STAGE_BYTES > OUT_BYTES ? STAGE_BYTES : OUT_BYTES];
  T (*sA)[BM * PITCH] = reinterpret_cast<T (*)[BM * PITCH]>(smem);
  T (*sB)[BN * PITCH] = reinterpret_cast<T (*)[BN * PITCH]>(smem + 2 * BM * PITCH * sizeof(T));

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int H = a.H, W = a.W, C = a.C, S = a.S, pad = a.pad, padw = a.padw;
  // the GEMM rows: the input grid for GM 0, else the Ho x Wo grid
  const int Ho = GM ? a.Ho : H, Wo = GM ? a.Wo : W;
  const int sd = GM ? a.stride : 1;
  const int M = a.nb * Ho * Wo;
  const int Min = a.nb * H * W;  // pixels of x
  const int K = a.R * S * C;
  // logical tile (row tile tm, column tile tn), column tiles fastest
  const int tlin = xcd_tile(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
  const int tm = tlin / gridDim.y, tn = tlin - tm * gridDim.y;
  const int m0 = tm * BM, n0 = tn * BN;
  const T* __restrict__ x = (const T*)a.x;
  const T* __restrict__ w = (const T*)a.w;

  // fixed per-thread chunk slots
  int a_row[A_PER], a_kc[A_PER], a_img[A_PER], a_h[A_PER], a_w[A_PER];
  bool a_slot[A_PER], a_valid[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    int q = tid + i * NT;
    a_slot[i] = q < A_CH;
    a_row[i] = q / CPR;
    a_kc[i] = q % CPR;
    int m = m0 + a_row[i];
    a_valid[i] = a_slot[i] && m < M;
    int mm = a_valid[i] ? m : 0;
    a_img[i] = mm / (Ho * Wo);
    int rem = mm - a_img[i] * Ho * Wo;
    a_h[i] = rem / Wo;
    a_w[i] = rem - a_h[i] * Wo;
  }
  int b_row[B_PER], b_kc[B_PER];
  bool b_slot[B_PER], b_valid[B_PER];
#pragma unroll
  for (int i = 0; i < B_PER; ++i) {
    int q = tid + i * NT;
    b_slot[i] = q < B_CH;
    b_row[i] = q / CPR;
    b_kc[i] = q % CPR;
    b_valid[i] = b_slot[i] && (n0 + b_row[i]) < a.N;
  }

  // Buffer-load addressing (16-byte chunk path): the input and weight views
  // are raw buffer resources whose loads return zeros past num_records, so a
  // chunk outside the image or past the channels is read from offset
  // OUT_OF_RANGE instead of being branched around.  Per thread: the byte
  // offset of each chunk's pixel, and one bit per filter row (column) telling
  // whether that row (column) of taps lands inside the image.
  constexpr uint32_t OUT_OF_RANGE = 0x80000000u;
  uint32_t a_off[A_PER], b_off[B_PER], a_hm[A_PER], a_wm[A_PER];
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)x, (short)0, (int)((((size_t)(Min - 1)) * a.ldx + C) * sizeof(T)), 0x00020000);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)w, (short)0, (int)((size_t)a.N * K * sizeof(T)), 0x00020000);
  if constexpr (!FLAT) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      // base pixel of the row's taps; a tap adds (r - pad, q - pad) (GM 0, 1) or
      // (-(r / sd), -(q / sd)) (GM 2); 32-bit wrap-around makes a base one row
      // past the image harmless, since only in-image taps use it
      const int bh = GM == 2 ? (a_h[i] + pad) / sd : a_h[i] * sd;
      const int bw = GM == 2 ? (a_w[i] + padw) / sd : a_w[i] * sd;
      a_off[i] = (uint32_t)((((size_t)(a_img[i] * H + bh) * W + bw) * a.ldx + a_kc[i] * VEC) *
                            sizeof(T));
      uint32_t hm = 0, wm = 0;
      if (a_valid[i]) {
        if constexpr (GM == 2) {
          for (int r = 0; r < a.R; ++r) {
            const int t = a_h[i] + pad - r;
            hm |= (uint32_t)(t >= 0 && t % sd == 0 && t / sd < H) << r;
          }
          for (int q = 0; q < S; ++q) {
            const int t = a_w[i] + padw - q;
            wm |= (uint32_t)(t >= 0 && t % sd == 0 && t / sd < W) << q;
          }
        } else {
          for (int r = 0; r < a.R; ++r)
            hm |= (uint32_t)((unsigned)(bh + r - pad) < (unsigned)H) << r;
          for (int q = 0; q < S; ++q)
            wm |= (uint32_t)((unsigned)(bw + q - padw) < (unsigned)W) << q;
        }
      }
      a_hm[i] = hm;
      a_wm[i] = wm;
    }
#pragma unroll
    for (int i = 0; i < B_PER; ++i)
      b_off[i] = b_valid[i] ? (uint32_t)(((size_t)(n0 + b_row[i]) * K + b_kc[i] * VEC) * sizeof(T))
                            : OUT_OF_RANGE;
  }

  const int nCB = FLAT ? 1 : (C + BK - 1) / BK;
  const int nk = FLAT ? (K + BK - 1) / BK : a.R * S * nCB;

  // PF register slots: the global loads of PF k-tiles are in flight at once.
  uint4 ra[PF][A_PER], rb[PF][B_PER];
  // position of the next k-tile to load (16-byte chunk path): filter row lr,
  // column lq, channel block lcb; advanced once per load, held at the last tile
  int lr = 0, lq = 0, lcb = 0, lrs = 0, loaded = 0;

  // slot indices are compile-time constants so the register ring is not spilled
  auto gload = [&](int kb, auto SLOT) __attribute__((always_inline)) {
    constexpr int slot = decltype(SLOT)::value;
    if constexpr (!FLAT) {
      (void)kb;
      const int crem = C - lcb * BK;  // channels left in this tap from this block on
      const int tr_ = GM == 2 ? -(lr / sd) : lr - pad;
      const int tq_ = GM == 2 ? -(lq / sd) : lq - padw;
      const int dx = ((tr_ * W + tq_) * a.ldx + lcb * BK) * (int)sizeof(T);
      const uint32_t dw = (uint32_t)((lrs * C + lcb * BK) * (int)sizeof(T));
#pragma unroll
      for (int i = 0; i < A_PER; ++i) {
        const bool ok = ((a_hm[i] >> lr) & (a_wm[i] >> lq) & 1u) && a_kc[i] * VEC < crem;
        const uint32_t off = ok ? a_off[i] + (uint32_t)dx : OUT_OF_RANGE;
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0);
        ra[slot][i] = make_uint4(v[0], v[1], v[2], v[3]);
      }
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        const bool ok = b_kc[i] * VEC < crem;
        const uint32_t off = ok ? b_off[i] + dw : OUT_OF_RANGE;
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(wr, (int)off, 0, 0);
        rb[slot][i] = make_uint4(v[0], v[1], v[2], v[3]);
      }
      // advance the cursor without branches (the loop body stays one block)
      const bool adv = ++loaded < nk;
      const bool wc = adv && lcb + 1 == nCB;
      const bool wq = wc && lq + 1 == S;
      lcb = wc ? 0 : lcb + (int)adv;
      lrs += (int)wc;
      lq = wq ? 0 : lq + (int)wc;
      lr += (int)wq;
    } else {
#pragma unroll
      for (int i = 0; i < A_PER; ++i) {
        T vals[VEC];
        // (r, s, c) of the chunk's first k, then stepped element by element
        const int kbase = kb * BK + a_kc[i] * VEC;
        int r = kbase / (S * C), s = (kbase / C) % S, c = kbase % C;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int k = kbase + e;
          T val = zero_elem<T>();
          if (a_valid[i] && k < K) {
            int hh, ww;
            bool in;
            if constexpr (GM == 2) {
              const int th = a_h[i] + pad - r, tw = a_w[i] + padw - s;
              in = th >= 0 && tw >= 0 && th % sd == 0 && tw % sd == 0;
              hh = th / sd;
              ww = tw / sd;
            } else {
              hh = a_h[i] * sd + r - pad;
              ww = a_w[i] * sd + s - padw;
              in = true;
            }
            if (in && hh >= 0 && hh < H && ww >= 0 && ww < W)
              val = x[((size_t)(a_img[i] * H + hh) * W + ww) * a.ldx + c];
          }
          vals[e] = val;
          if (++c == C) {
            c = 0;
            if (++s == S) {
              s = 0;
              ++r;
            }
          }
        }
        ra[slot][i] = pack_chunk<T>(vals);
      }
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        T vals[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          int k = kb * BK + b_kc[i] * VEC + e;
          vals[e] = (b_valid[i] && k < K) ? w[(size_t)(n0 + b_row[i]) * K + k] : zero_elem<T>();
        }
        rb[slot][i] = pack_chunk<T>(vals);
      }
    }
  };
  // LDS element offset of each slot's chunk; a slot past the tile writes into
  // the row padding (never read), so the stores need no branches
  int a_lds[A_PER], b_lds[B_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i)
    a_lds[i] = a_slot[i] ? a_row[i] * PITCH + a_kc[i] * VEC : ((tid + i * NT - A_CH) % BM) * PITCH + BK;
#pragma unroll
  for (int i = 0; i < B_PER; ++i)
    b_lds[i] = b_slot[i] ? b_row[i] * PITCH + b_kc[i] * VEC : ((tid + i * NT - B_CH) % BN) * PITCH + BK;
  auto lstore = [&](auto SLOT, int buf) __attribute__((always_inline)) {
    constexpr int slot = decltype(SLOT)::value;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) *reinterpret_cast<uint4*>(&sA[buf][a_lds[i]]) = ra[slot][i];
#pragma unroll
    for (int i = 0; i < B_PER; ++i) *reinterpret_cast<uint4*>(&sB[buf][b_lds[i]]) = rb[slot][i];
  };

  constexpr int TM2 = M32 ? WTM / 32 : 1, TN2 = M32 ? WTN / 32 : 1;
  typename MTT::acc_t acc[M32 ? 1 : TM][M32 ? 1 : TN];
  f32x16_t acc2[TM2][TN2];
  if constexpr (M32) {
#pragma unroll
    for (int i = 0; i < TM2; ++i)
#pragma unroll
      for (int j = 0; j < TN2; ++j)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc2[i][j][q] = 0.f;
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[i][j][q] = 0;
  }

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const T* A = sA[buf];
    const T* B = sB[buf];
    if constexpr (M32) {
      // A fragment: lane l holds row l % 32, k = 8 * (l / 32) .. + 8 of a 16-deep step
#pragma unroll
      for (int kk = 0; kk < BK / 16; ++kk) {
        bf16x8_t af[TM2], bfv[TN2];
#pragma unroll
        for (int i = 0; i < TM2; ++i)
          af[i] = *reinterpret_cast<const bf16x8_t*>(
              &A[(wm * WTM + i * 32 + (lane & 31)) * PITCH + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
        for (int j = 0; j < TN2; ++j)
          bfv[j] = *reinterpret_cast<const bf16x8_t*>(
              &B[(wn * WTN + j * 32 + (lane & 31)) * PITCH + kk * 16 + (lane >> 5) * 8]);
#pragma unroll
        for (int i = 0; i < TM2; ++i)
#pragma unroll
          for (int j = 0; j < TN2; ++j)
            acc2[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfv[j], acc2[i][j], 0, 0, 0);
      }
    } else if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8_t af[TM], bfv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = *reinterpret_cast<const bf16x8_t*>(
              &A[(wm * WTM + i * 16 + (lane & 15)) * PITCH + ks * 32 + (lane >> 4) * 8]);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfv[j] = *reinterpret_cast<const bf16x8_t*>(
              &B[(wn * WTN + j * 16 + (lane & 15)) * PITCH + ks * 32 + (lane >> 4) * 8]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfv[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < BK / 4; ++kk) {
        double af[TM], bfv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = (double)A[(wm * WTM + i * 16 + (lane & 15)) * PITCH + kk * 4 + (lane >> 4)];
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfv[j] = (double)B[(wn * WTN + j * 16 + (lane & 15)) * PITCH + kk * 4 + (lane >> 4)];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  // k-tile j is loaded into register slot j % PF, PF tiles ahead of its use,
  // and staged into LDS buffer j & 1 one step ahead
  // Loads are issued unconditionally (the last tile is re-read past the end)
  // so that the only waits are for the tile about to be staged.
  static_for<0, PF>([&](auto J) __attribute__((always_inline)) {
    gload(min((int)decltype(J)::value, nk - 1), J);
  });
  lstore(std::integral_constant<int, 0>{}, 0);
  __syncthreads();
  int kb0 = 0;
  for (; kb0 + PF <= nk; kb0 += PF) {
    static_for<0, PF>([&](auto U) __attribute__((always_inline)) {
      constexpr int u = decltype(U)::value;
      const int kb = kb0 + u;
      // MFMAs on tile kb first, then refill slot u (tile kb, already in LDS)
      // with tile kb + PF and stage tile kb + 1 into the other buffer (last
      // read one step ago); past the end both repeat the last tile harmlessly
      compute(kb & 1);
      gload(min(kb + PF, nk - 1), U);
      lstore(std::integral_constant<int, (u + 1) % PF>{}, (kb + 1) & 1);
      __syncthreads();
    });
  }
  static_for<0, PF>([&](auto U) __attribute__((always_inline)) {
    constexpr int u = decltype(U)::value;
    const int kb = kb0 + u;
    if (kb < nk) {
      compute(kb & 1);
      if (kb + 1 < nk) lstore(std::integral_constant<int, (u + 1) % PF>{}, (kb + 1) & 1);
      __syncthreads();
    }
  });

  T* __restrict__ y = (T*)a.y;
  const T* __restrict__ mask = (const T*)a.mask;
  if constexpr (sizeof(T) == 2) {
    // epilogue (bf16): stage the fp32 tile in LDS, then each thread finishes
    // 8-column chunks of a row (bias, ReLU, mask, accumulate, round once) with
    // 16-byte loads and stores, and leaves the stored values in LDS for the
    // batch-norm column statistics.  The main loop ended with a barrier, so
    // the operand tiles are free.
    float* ot = reinterpret_cast<float*>(smem);
    if constexpr (M32) {
      // 32x32 result: lane l, register r holds row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
#pragma unroll
      for (int i = 0; i < TM2; ++i)
#pragma unroll
        for (int j = 0; j < TN2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            ot[(wm * WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * OPITCH + wn * WTN +
               j * 32 + (lane & 31)] = acc2[i][j][r];
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            ot[(wm * WTM + i * 16 + MTT::out_row(lane, q)) * OPITCH + wn * WTN + j * 16 + (lane & 15)] =
                acc[i][j][q];
    }
    __syncthreads();
    conv_epilogue_bf16<BM, BN, NT, OPITCH>(a, ot, tid, m0, n0, tm, M, gridDim.x);
  } else {
    // epilogue (fp32 storage): bias, ReLU, mask, accumulate, round once on store
    constexpr int NCOL = M32 ? TN2 : TN;  // column groups per lane
    double cs[NCOL], cq[NCOL];  // column sums of the stored values (batch-norm statistics)
#pragma unroll
    for (int j = 0; j < NCOL; ++j) cs[j] = cq[j] = 0.0;
    auto emit = [&](double acc_v, int m, int n, int j) __attribute__((always_inline)) {
      if (m < M && n < a.N) {
        double v = acc_v;
        if (a.bias) v += (double)a.bias[n];
        if (a.relu) v = v > 0.0 ? v : 0.0;
        if (mask && !(ldd(mask + (size_t)m * a.ldm + n) > 0.0)) v = 0.0;
        T* p = y + (size_t)m * a.ldy + n;
        if (a.accumulate) v += ldd(p);
        std_(p, v);
        if (a.stat_part) {
          double sv = ldd(p);  // the stored (rounded) value, as the statistics see it
          cs[j] += sv;
          cq[j] += sv * sv;
        }
      }
    };
    if constexpr (M32) {
      // 32x32 result: lane l, register r holds row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
#pragma unroll
      for (int i = 0; i < TM2; ++i)
#pragma unroll
        for (int j = 0; j < TN2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            emit((double)acc2[i][j][r], m0 + wm * WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3),
                 n0 + wn * WTN + j * 32 + (lane & 31), j);
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            emit((double)acc[i][j][q], m0 + wm * WTM + i * 16 + MTT::out_row(lane, q),
                 n0 + wn * WTN + j * 16 + (lane & 15), j);
    }
    if (a.stat_part) {
      // lanes that hold the same column add in a fixed butterfly order
      constexpr int CW = M32 ? 32 : 16;  // columns per group
#pragma unroll
      for (int j = 0; j < NCOL; ++j) {
        if constexpr (!M32) {
          cs[j] += __shfl_xor(cs[j], 16, 64);
          cq[j] += __shfl_xor(cq[j], 16, 64);
        }
        cs[j] += __shfl_xor(cs[j], 32, 64);
        cq[j] += __shfl_xor(cq[j], 32, 64);
      }
      __shared__ double red[WM][2][BN];
      if (lane < CW) {
#pragma unroll
        for (int j = 0; j < NCOL; ++j) {
          red[wm][0][wn * WTN + j * CW + lane] = cs[j];
          red[wm][1][wn * WTN + j * CW + lane] = cq[j];
        }
      }
      __syncthreads();
      for (int col = tid; col < BN; col += NT) {
        int n = n0 + col;
        if (n >= a.N) continue;
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int w = 0; w < WM; ++w) {
          s0 += red[w][0][col];
          s1 += red[w][1][col];
        }
        a.stat_part[((size_t)n * 2 + 0) * gridDim.x + tm] = s0;
        a.stat_part[((size_t)n * 2 + 1) * gridDim.x + tm] = s1;
      }
    }
  }
}

// ============================================================================
// weight-gradient GEMM with split reduction over pixels
// ============================================================================
// bf16: LDS tiles are [row][pixel] (pixel-contiguous) so the MFMA operand
// fragments are 16-byte reads; the global chunks run along channels, so each
// thread loads two pixels and interleaves them into 32-bit pairs on the way in.
// fp32/fp64: one element per lane per MFMA, so the natural [pixel][row] layout
// is read directly.
template <typename T> struct WG;
template <> struct WG<bf16_t> {
  static constexpr int BKm = 32;
};
template <> struct WG<float> {
  static constexpr int BKm = 16;
};

template <typename T, int BM, int BN, int WM, int WN, bool FLAT>
__global__ __launch_bounds__(256) void k_wgrad(WgradArgs a) {
  using MTT = MT<T>;
  constexpr int VEC = MTT::VEC;
  constexpr int BKm = WG<T>::BKm;
  constexpr bool BF = sizeof(T) == 2;
  // LDS geometry
  constexpr int PA = BF ? (BKm + 8) : (BM + 16);  // pitch of A tile rows
  constexpr int PB = BF ? (BKm + 8) : (BN + 16);
  constexpr int SA = BF ? BM * PA : BKm * PA;     // elements per buffer
  constexpr int SB = BF ? BN * PB : BKm * PB;
  __shared__ __align__(16) T sA[2][SA];
  __shared__ __align__(16) T sB[2][SB];
  constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
  static_assert(WM * WN == 4, "four waves");
  // load tasks: bf16: (pixel pair, 8-channel chunk); fp32: (pixel, 4-channel chunk)
  constexpr int A_T = BF ? (BKm / 2) * (BM / VEC) : BKm * (BM / VEC);
  constexpr int B_T = BF ? (BKm / 2) * (BN / VEC) : BKm * (BN / VEC);
  constexpr int A_PER = (A_T + 255) / 256, B_PER = (B_T + 255) / 256;
  constexpr int RPT = BF ? 2 : 1;  // pixels per task

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int H = a.H, W = a.W, C = a.C, S = a.S, pad = a.pad, padw = a.padw, N = a.N;
  // dz pixels: the input grid, or the Ho x Wo grid of a strided or unpadded
  // convolution
  const int sd = a.stride > 1 ? a.stride : 1;
  const int Wo = a.Ho > 0 ? a.Wo : W;
  const int HW = (a.Ho > 0 ? a.Ho : H) * Wo;
  const int M = a.nb * HW;
  const int K = a.R * S * C;
  const int n0 = blockIdx.x * BM, k0 = blockIdx.y * BN;
  const int mps = ((M + a.splits - 1) / a.splits + BKm - 1) / BKm * BKm;
  const int mbeg = blockIdx.z * mps;
  const int mend = min(M, mbeg + mps);
  const T* __restrict__ dz = (const T*)a.dz;
  const T* __restrict__ x = (const T*)a.x;
  const bool dz_vec = (a.lddz % VEC) == 0 && (reinterpret_cast<uintptr_t>(a.dz) % 16) == 0;

  // task geometry (fixed over the pixel loop)
  int a_p[A_PER], a_c[A_PER];
  bool a_slot[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    int q = tid + i * 256;
    a_slot[i] = q < A_T;
    a_c[i] = q % (BM / VEC);   // channel chunk (output-channel dim)
    a_p[i] = q / (BM / VEC);   // pixel (pair) index
  }
  int b_p[B_PER], b_c[B_PER], b_r[B_PER], b_s[B_PER], b_ch[B_PER];
  bool b_slot[B_PER], b_kok[B_PER];
#pragma unroll
  for (int i = 0; i < B_PER; ++i) {
    int q = tid + i * 256;
    b_slot[i] = q < B_T;
    b_c[i] = q % (BN / VEC);
    b_p[i] = q / (BN / VEC);
    int kk = k0 + b_c[i] * VEC;
    b_kok[i] = kk < K;
    // filter position and channel of the chunk's first k (the flat gather
    // steps through the chunk from there)
    int rs = kk / C;
    b_ch[i] = kk - rs * C;
    b_r[i] = rs / S;
    b_s[i] = rs - b_r[i] * S;
  }

  uint4 ra[A_PER][RPT], rb[B_PER][RPT];

  auto gload = [&](int mb) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
#pragma unroll
      for (int u = 0; u < RPT; ++u) {
        int m = mb + a_p[i] * RPT + u;
        int n = n0 + a_c[i] * VEC;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (a_slot[i] && m < mend && n < N) {
          const T* src = dz + (size_t)m * a.lddz + n;
          if (dz_vec && n + VEC <= N) {
            v = *reinterpret_cast<const uint4*>(src);
          } else {
            T vals[VEC];
#pragma unroll
            for (int e = 0; e < VEC; ++e) vals[e] = (n + e < N) ? src[e] : zero_elem<T>();
            v = pack_chunk<T>(vals);
          }
        }
        ra[i][u] = v;
      }
#pragma unroll
    for (int i = 0; i < B_PER; ++i)
#pragma unroll
      for (int u = 0; u < RPT; ++u) {
        int m = mb + b_p[i] * RPT + u;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (b_slot[i] && m < mend) {
          int img = m / HW, rem = m - img * HW, h = rem / Wo, ww0 = rem - h * Wo;
          h *= sd;
          ww0 *= sd;
          if constexpr (!FLAT) {
            int hh = h + b_r[i] - pad, ww = ww0 + b_s[i] - padw;
            if (b_kok[i] && hh >= 0 && hh < H && ww >= 0 && ww < W)
              v = *reinterpret_cast<const uint4*>(x + ((size_t)(img * H + hh) * W + ww) * a.ldx + b_ch[i]);
          } else {
            T vals[VEC];
            int r = b_r[i], s = b_s[i], c = b_ch[i];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
              int k = k0 + b_c[i] * VEC + e;
              T val = zero_elem<T>();
              if (k < K) {
                int hh = h + r - pad, ww = ww0 + s - padw;
                if (hh >= 0 && hh < H && ww >= 0 && ww < W)
                  val = x[((size_t)(img * H + hh) * W + ww) * a.ldx + c];
              }
              vals[e] = val;
              if (++c == C) {
                c = 0;
                if (++s == S) {
                  s = 0;
                  ++r;
                }
              }
            }
            v = pack_chunk<T>(vals);
          }
        }
        rb[i][u] = v;
      }
  };

  auto lstore = [&](int buf) {
    if constexpr (BF) {
      // interleave two pixels: word e of row (chunk*8 + e) holds (pixel 2p, pixel 2p+1)
#pragma unroll
      for (int i = 0; i < A_PER; ++i) {
        if (!a_slot[i]) continue;
        const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&ra[i][0]);
        const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&ra[i][1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint32_t lo = (r0[j] & 0xffffu) | (r1[j] << 16);
          uint32_t hi = (r0[j] >> 16) | (r1[j] & 0xffff0000u);
          int row = a_c[i] * VEC + 2 * j;
          *reinterpret_cast<uint32_t*>(&sA[buf][row * PA + 2 * a_p[i]]) = lo;
          *reinterpret_cast<uint32_t*>(&sA[buf][(row + 1) * PA + 2 * a_p[i]]) = hi;
        }
      }
#pragma unroll
      for (int i = 0; i < B_PER; ++i) {
        if (!b_slot[i]) continue;
        const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&rb[i][0]);
        const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&rb[i][1]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint32_t lo = (r0[j] & 0xffffu) | (r1[j] << 16);
          uint32_t hi = (r0[j] >> 16) | (r1[j] & 0xffff0000u);
          int row = b_c[i] * VEC + 2 * j;
          *reinterpret_cast<uint32_t*>(&sB[buf][row * PB + 2 * b_p[i]]) = lo;
          *reinterpret_cast<uint32_t*>(&sB[buf][(row + 1) * PB + 2 * b_p[i]]) = hi;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < A_PER; ++i)
        if (a_slot[i]) *reinterpret_cast<uint4*>(&sA[buf][a_p[i] * PA + a_c[i] * VEC]) = ra[i][0];
#pragma unroll
      for (int i = 0; i < B_PER; ++i)
        if (b_slot[i]) *reinterpret_cast<uint4*>(&sB[buf][b_p[i] * PB + b_c[i] * VEC]) = rb[i][0];
    }
  };

  typename MTT::acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[i][j][q] = 0;

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const T* A = sA[buf];
    const T* B = sB[buf];
    if constexpr (BF) {
      bf16x8_t af[TM], bfv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(&A[(wm * WTM + i * 16 + (lane & 15)) * PA + (lane >> 4) * 8]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfv[j] = *reinterpret_cast<const bf16x8_t*>(&B[(wn * WTN + j * 16 + (lane & 15)) * PB + (lane >> 4) * 8]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfv[j], acc[i][j], 0, 0, 0);
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        double af[TM], bfv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[i] = (double)A[(kk * 4 + (lane >> 4)) * PA + wm * WTM + i * 16 + (lane & 15)];
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfv[j] = (double)B[(kk * 4 + (lane >> 4)) * PB + wn * WTN + j * 16 + (lane & 15)];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  const int nsteps = mend > mbeg ? (mend - mbeg + BKm - 1) / BKm : 0;
  if (nsteps > 0) {
    gload(mbeg);
    lstore(0);
  }
  __syncthreads();
  for (int st = 0; st < nsteps; ++st) {
    const bool more = st + 1 < nsteps;
    if (more) gload(mbeg + (st + 1) * BKm);
    compute(st & 1);
    if (more) lstore((st + 1) & 1);
    __syncthreads();
  }

  typename MTT::part_t* part = (typename MTT::part_t*)a.part + (size_t)blockIdx.z * N * K;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int n = n0 + wm * WTM + i * 16 + MTT::out_row(lane, q);
        int k = k0 + wn * WTN + j * 16 + (lane & 15);
        if (n < N && k < K) part[(size_t)n * K + k] = acc[i][j][q];
      }
}


// bf16 weight gradient, 16-byte chunk path (channels, output channels and row
// strides multiples of 8, views below 2 GiB), 32x32 wave tiles.  The operands
// load through raw buffer resources (out-of-range offsets read zeros),
// addresses advance by a scalar per step, each thread tracks the image row /
// column of its pixel incrementally, and PF steps of loads are in flight.
// The reduction runs over pixels, which are the rows of both operands in
// memory, while an MFMA fragment holds 8 consecutive pixels of one column: the
// tiles therefore sit in LDS as loaded (one row per pixel, 16-byte stores) and
// the fragments are read with gfx950's transposing LDS read.  Interleaving
// pixel pairs into column-major rows on the way into LDS instead (two
// permutes and two 4-byte LDS stores per 16 loaded bytes) was 30% slower on
// the 3x3 and 5x5 stage shapes (3x3 64 -> 96: 35.4 -> 24.6 us with the split
// reduction), with the same bits.
// GRID: dz lives on the Ho x Wo grid of a strided or unpadded convolution (or
// the rows and columns pad differently); each pixel then tracks its image, row
// and column and addresses x at (ho*stride + r - pad, wo*stride + q - padw)
template <int BM, int BN, int WM, int WN, int PF, bool GRID>
__global__ __launch_bounds__(256) void k_wgrad_t(WgradArgs a) {
  using T = bf16_t;
  // 64 pixels per step: four 32x32x16 MFMAs per wave between barriers (32 took
  // 4-8% longer on the stage shapes)
  constexpr int VEC = 8, BKm = 64, RPT = 1;
  // rows = pixels, as loaded; a row pitch of 32 bytes over the tile width puts
  // the four rows one transposing read touches in disjoint banks
  constexpr int PA = BM + 16, PB = BN + 16;
  __shared__ __align__(16) T sA[2][BKm * PA];
  __shared__ __align__(16) T sB[2][BKm * PB];
  constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 16, TN = WTN / 16;
  static_assert(WM * WN == 4, "four waves");
  constexpr int A_T = BKm * (BM / VEC), B_T = BKm * (BN / VEC);
  constexpr int A_PER = (A_T + 255) / 256, B_PER = (B_T + 255) / 256;
  constexpr uint32_t OUT_OF_RANGE = 0x80000000u;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int H = a.H, W = a.W, C = a.C, S = a.S, pad = a.pad, N = a.N;
  const int padw = GRID ? a.padw : pad;
  const int sd = GRID && a.stride > 1 ? a.stride : 1;
  const int Ho = GRID && a.Ho > 0 ? a.Ho : H, Wo = GRID && a.Ho > 0 ? a.Wo : W;
  const int M = a.nb * Ho * Wo;    // dz pixels
  const int Min = a.nb * H * W;    // x pixels
  const int K = a.R * S * C;
  const int n0 = blockIdx.x * BM, k0 = blockIdx.y * BN;
  const int mps = ((M + a.splits - 1) / a.splits + BKm - 1) / BKm * BKm;
  const int mbeg = blockIdx.z * mps;
  const int mend = min(M, mbeg + mps);
  const __amdgpu_buffer_rsrc_t dr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.dz, (short)0, (int)((((size_t)(M - 1)) * a.lddz + N) * sizeof(T)), 0x00020000);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.x, (short)0, (int)((((size_t)(Min - 1)) * a.ldx + C) * sizeof(T)), 0x00020000);

  // A tasks (dz): pixel pair p, output-channel chunk c
  int a_p[A_PER], a_c[A_PER];
  uint32_t a_off[A_PER];
  bool a_slot[A_PER], a_nok[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    const int q = tid + i * 256;
    a_slot[i] = q < A_T;
    a_c[i] = q % (BM / VEC);
    a_p[i] = q / (BM / VEC);
    const int n = n0 + a_c[i] * VEC;
    a_nok[i] = a_slot[i] && n < N;
    a_off[i] = (uint32_t)((((size_t)mbeg + a_p[i] * RPT) * a.lddz + n) * sizeof(T));
  }
  // B tasks (x): pixel pair p, reduction chunk (tap r, s, channel ch)
  int b_p[B_PER], b_c[B_PER], b_r[B_PER], b_s[B_PER], b_ch[B_PER];
  int b_h[B_PER][RPT], b_w[B_PER][RPT], b_img[B_PER][RPT];
  uint32_t b_off[B_PER];
  bool b_slot[B_PER], b_kok[B_PER];
#pragma unroll
  for (int i = 0; i < B_PER; ++i) {
    const int q = tid + i * 256;
    b_slot[i] = q < B_T;
    b_c[i] = q % (BN / VEC);
    b_p[i] = q / (BN / VEC);
    const int kk = k0 + b_c[i] * VEC;
    b_kok[i] = b_slot[i] && kk < K;
    const int rs = b_kok[i] ? kk / C : 0, ch = b_kok[i] ? kk - rs * C : 0;
    b_r[i] = rs / S;
    b_s[i] = rs - b_r[i] * S;
    b_ch[i] = ch;
    // byte offset of (first pixel of the pair at step 0, shifted by the tap)
    const long long pix = (long long)mbeg + b_p[i] * RPT + (b_r[i] - pad) * W + (b_s[i] - pad);
    b_off[i] = GRID ? 0u : (uint32_t)((pix * a.ldx + ch) * (long long)sizeof(T));
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int m = mbeg + b_p[i] * RPT + u;
      const int rem = m % (Ho * Wo);
      b_img[i][u] = m / (Ho * Wo);
      b_h[i][u] = rem / Wo;
      b_w[i][u] = rem - b_h[i][u] * Wo;
    }
  }

  uint4 ra[PF][A_PER][RPT], rb[PF][B_PER][RPT];
  int loaded = 0;  // steps loaded so far

  auto gload = [&](auto SLOT) __attribute__((always_inline)) {
    constexpr int slot = decltype(SLOT)::value;
    const int mb = loaded * BKm;  // pixel offset of this step from mbeg
    const int left = mend - mbeg - mb;
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
#pragma unroll
      for (int u = 0; u < RPT; ++u) {
        const bool ok = a_nok[i] && a_p[i] * RPT + u < left;
        const uint32_t off =
            ok ? a_off[i] + (uint32_t)(((size_t)mb + u) * a.lddz * sizeof(T)) : OUT_OF_RANGE;
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(dr, (int)off, 0, 0);
        ra[slot][i][u] = make_uint4(v[0], v[1], v[2], v[3]);
      }
#pragma unroll
    for (int i = 0; i < B_PER; ++i)
#pragma unroll
      for (int u = 0; u < RPT; ++u) {
        const int hh = b_h[i][u] * sd + b_r[i] - pad, ww = b_w[i][u] * sd + b_s[i] - padw;
        const bool ok = b_kok[i] && b_p[i] * RPT + u < left && (unsigned)hh < (unsigned)H &&
                        (unsigned)ww < (unsigned)W;
        uint32_t off;
        if constexpr (GRID)
          off = ok ? (uint32_t)(((((size_t)b_img[i][u] * H + hh) * W + ww) * a.ldx + b_ch[i]) * sizeof(T))
                   : OUT_OF_RANGE;
        else
          off = ok ? b_off[i] + (uint32_t)(((size_t)mb + u) * a.ldx * sizeof(T)) : OUT_OF_RANGE;
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0);
        rb[slot][i][u] = make_uint4(v[0], v[1], v[2], v[3]);
        // advance this pixel by one step
        int w2 = b_w[i][u] + BKm, h2 = b_h[i][u];
        while (w2 >= Wo) {
          w2 -= Wo;
          if (++h2 == Ho) {
            h2 = 0;
            if constexpr (GRID) ++b_img[i][u];
          }
        }
        b_w[i][u] = w2;
        b_h[i][u] = h2;
      }
    ++loaded;
  };

  // each task's 16 bytes (8 channels of one pixel) go to its pixel's row as
  // loaded: no interleaving
  auto lstore = [&](auto SLOT, int buf) __attribute__((always_inline)) {
    constexpr int slot = decltype(SLOT)::value;
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
      if (a_slot[i]) *reinterpret_cast<uint4*>(&sA[buf][a_p[i] * PA + a_c[i] * VEC]) = ra[slot][i][0];
#pragma unroll
    for (int i = 0; i < B_PER; ++i)
      if (b_slot[i]) *reinterpret_cast<uint4*>(&sB[buf][b_p[i] * PB + b_c[i] * VEC]) = rb[slot][i][0];
  };

  // wave tiles that are multiples of 32 use v_mfma_f32_32x32x16_bf16
  constexpr bool M32 = WTM % 32 == 0 && WTN % 32 == 0;
  static_assert(M32, "32x32 wave tiles");
  constexpr int TM2 = M32 ? WTM / 32 : 1, TN2 = M32 ? WTN / 32 : 1;
  f32x4_t acc[M32 ? 1 : TM][M32 ? 1 : TN];
  f32x16_t acc2[TM2][TN2];
#pragma unroll
  for (int i = 0; i < (M32 ? 1 : TM); ++i)
#pragma unroll
    for (int j = 0; j < (M32 ? 1 : TN); ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[i][j][q] = 0.f;
#pragma unroll
  for (int i = 0; i < TM2; ++i)
#pragma unroll
    for (int j = 0; j < TN2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc2[i][j][q] = 0.f;

  // MFMA fragments straight from the pixel-major tiles with gfx950's
  // transposing LDS read: in each group of 16 lanes, output e (0..3) of lane i
  // is element i % 4 of the 8 bytes that lane 4 e + i / 4 of the group
  // addressed.  A 32x32x16 fragment (lane l: row l % 32, pixels 8 (l / 32) ..
  // + 8 of the 16-pixel slice) is two such reads: lane j of a group addresses
  // pixel 8 (l / 32) + j / 4 (+ 4 for the second read), columns
  // 16 ((l % 32) / 16) + 4 (j % 4) .. + 4 of the wave's 32.
  const int tr_px = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane & 31) >> 4) + 4 * (lane & 3);
  auto tr_frag = [&](const T* base, int pitch, int col0, int px0) __attribute__((always_inline)) {
    typedef short v4i16 __attribute__((ext_vector_type(4)));
    const T* p = base + (px0 + tr_px) * pitch + col0 + tr_col;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(p));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4i16*)(p + 4 * pitch));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, v);
  };
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const T* A = sA[buf];
    const T* B = sB[buf];
#pragma unroll
    for (int kk = 0; kk < BKm / 16; ++kk) {
      bf16x8_t af[TM2], bfv[TN2];
#pragma unroll
      for (int i = 0; i < TM2; ++i) af[i] = tr_frag(A, PA, wm * WTM + i * 32, kk * 16);
#pragma unroll
      for (int j = 0; j < TN2; ++j) bfv[j] = tr_frag(B, PB, wn * WTN + j * 32, kk * 16);
#pragma unroll
      for (int i = 0; i < TM2; ++i)
#pragma unroll
        for (int j = 0; j < TN2; ++j)
          acc2[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfv[j], acc2[i][j], 0, 0, 0);
    }
  };

  const int nsteps = mend > mbeg ? (mend - mbeg + BKm - 1) / BKm : 0;
  if (nsteps > 0) {
    // step j loads into slot j % PF; the last step is re-read past the end
    static_for<0, PF>([&](auto J) __attribute__((always_inline)) {
      if (decltype(J)::value >= nsteps) loaded = nsteps - 1;
      gload(J);
    });
    lstore(std::integral_constant<int, 0>{}, 0);
    __syncthreads();
    int st0 = 0;
    for (; st0 + PF <= nsteps; st0 += PF) {
      static_for<0, PF>([&](auto U) __attribute__((always_inline)) {
        constexpr int u = decltype(U)::value;
        const int st = st0 + u;
        if (st + PF >= nsteps) loaded = nsteps - 1;
        gload(U);
        compute(st & 1);
        if (st + 1 < nsteps) lstore(std::integral_constant<int, (u + 1) % PF>{}, (st + 1) & 1);
        __syncthreads();
      });
    }
    static_for<0, PF>([&](auto U) __attribute__((always_inline)) {
      constexpr int u = decltype(U)::value;
      const int st = st0 + u;
      if (st < nsteps) {
        compute(st & 1);
        if (st + 1 < nsteps) lstore(std::integral_constant<int, (u + 1) % PF>{}, (st + 1) & 1);
        __syncthreads();
      }
    });
  }

  float* part = (float*)a.part + (size_t)blockIdx.z * N * K;
  // one split: grad (+)= the tile, the one addition the split reduction
  // would make; row n goes to its sibling's accumulator when rows are split
  auto put = [&](int n, int k, float v) __attribute__((always_inline)) {
    if (n >= N || k >= K) return;
    if (!a.direct) {
      part[(size_t)n * K + k] = v;
      return;
    }
    float* g = a.grad;
    int r = n;
    for (int j = 0; j < a.nseg; ++j)
      if (n >= a.seg_row0[j] && n < a.seg_row0[j + 1]) {
        g = a.seg_grad[j];
        r = n - a.seg_row0[j];
      }
    float* gi = g + (size_t)r * K + k;
    *gi = (float)((double)*gi + (double)v);  // as the split reduction adds
  };
  if constexpr (M32) {
#pragma unroll
    for (int i = 0; i < TM2; ++i)
#pragma unroll
      for (int j = 0; j < TN2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          put(n0 + wm * WTM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3),
              k0 + wn * WTN + j * 32 + (lane & 31), acc2[i][j][r]);
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          put(n0 + wm * WTM + i * 16 + MT<T>::out_row(lane, q), k0 + wn * WTN + j * 16 + (lane & 15),
              acc[i][j][q]);
  }
}

// grad[i] += sum over splits of part[z][i], splits added in order z = 0, 1, ...;
// each thread owns four consecutive outputs so the partial reads are 16-32 B
// Destination rows of the weight gradient: one accumulator, or several
// consecutive row ranges each with its own (sibling layers sharing a launch).
struct GradDst {
  int nseg;
  int64_t base[GATHER_MAX_SEGS + 1];  // flat element index where segment j starts
  float* ptr[GATHER_MAX_SEGS];
};

XP_DEV float* grad_at(const GradDst& d, int64_t i, int64_t* seg_end) {
  int j = 0;
  while (j + 1 < d.nseg && i >= d.base[j + 1]) ++j;
  *seg_end = d.base[j + 1];
  return d.ptr[j] + (i - d.base[j]);
}

// Threads are (quad, split group): the G groups of a quad of 4 consecutive
// elements add splits g, g + G, g + 2G, ... in order, then the first group
// adds the G group sums in group order and accumulates into grad (fixed order
// throughout: bit-reproducible).
constexpr int SPLIT_GROUPS = 8;
template <typename P>
__global__ __launch_bounds__(256) void k_split_reduce(const P* __restrict__ part, int splits,
                                                       int64_t count, GradDst dst) {
  constexpr int G = SPLIT_GROUPS, QPB = 256 / G;
  __shared__ double sh[G][QPB][4];
  const int qi = threadIdx.x % QPB, g = threadIdx.x / QPB;
  const int64_t q = ((int64_t)blockIdx.x * QPB + qi) * 4;
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  if (q + 4 <= count) {
#pragma unroll 4
    for (int z = g; z < splits; z += G) {
      const P* p = part + (size_t)z * count + q;
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] += (double)p[e];
    }
  } else if (q < count) {
    for (int z = g; z < splits; z += G)
      for (int e = 0; q + e < count; ++e) s[e] += (double)part[(size_t)z * count + q + e];
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) sh[g][qi][e] = s[e];
  __syncthreads();
  if (g != 0 || q >= count) return;
  double t[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    t[e] = sh[0][qi][e];
#pragma unroll
    for (int k = 1; k < G; ++k) t[e] += sh[k][qi][e];
  }
  int64_t seg_end = 0;
  float* gp = grad_at(dst, q, &seg_end);
  if (q + 4 <= seg_end) {
#pragma unroll
    for (int e = 0; e < 4; ++e) gp[e] = (float)((double)gp[e] + t[e]);
  } else {
    for (int e = 0; e < 4 && q + e < count; ++e) {
      float* gi = grad_at(dst, q + e, &seg_end);
      *gi = (float)((double)*gi + t[e]);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_gather(GatherArgs a) {
  for (int j = 0; j < a.nseg; ++j) {
    const T* src = (const T*)a.src[j];
    T* dst = (T*)a.dst[j];
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.count[j];
         i += (int64_t)gridDim.x * blockDim.x)
      dst[i] = src[i];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_flip_set(FlipSet f) {
  const int q = blockIdx.y;
  const T* __restrict__ w = (const T*)f.w[q];
  T* __restrict__ wd = (T*)f.wd[q];
  const int N = f.N[q], R = f.R[q], S = f.S[q], C = f.C[q], flip = f.flip[q];
  const int64_t total = (int64_t)N * R * S * C;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    // i indexes wd[c][r][s][n]
    int n = (int)(i % N);
    int64_t t = i / N;
    int s = (int)(t % S);
    t /= S;
    int r = (int)(t % R);
    int c = (int)(t / R);
    const int rr = flip ? R - 1 - r : r, ss = flip ? S - 1 - s : s;
    wd[i] = w[(((int64_t)n * R + rr) * S + ss) * C + c];
  }
}

// ============================================================================
// host launchers
// ============================================================================
// The bf16 stage depth minimises the zero padding of each tap's channel run
// while keeping at least four pipeline stages when possible.
static int pick_ks_bf16(int C, int taps) {
  // score: (at least 4 stages, least padding, then larger KS if >= 4 stages,
  // else more stages)
  int best = 1, b_ok = -1, b_pad = 0, b_tie = 0;
  for (int ks : {4, 2, 1}) {
    int bk = 32 * ks;
    int per_tap = (C + bk - 1) / bk;
    int pad = per_tap * bk;
    int ok = per_tap * taps >= 4;
    int tie = ok ? ks : -ks;
    if (ok > b_ok || (ok == b_ok && (pad < b_pad || (pad == b_pad && tie > b_tie)))) {
      best = ks;
      b_ok = ok;
      b_pad = pad;
      b_tie = tie;
    }
  }
  return best;
}

template <typename T> static const char* tname() { return sizeof(T) == 2 ? "bf16" : "f32"; }

template <typename T, int BM, int BN, int WM, int WN, bool FLAT, int KS = 0, int PF = 0, int GM = 0>
static const char* kname(const char* base) {
  static char buf[96];
  static bool init = false;
  if (!init) {
    if (KS && GM)
      snprintf(buf, sizeof buf, "%s<%s,%d,%d,%d,%d,%s,%d,%d,%s>", base, tname<T>(), BM, BN, WM, WN,
               FLAT ? "true" : "false", KS, PF, GM == 1 ? "strided" : "strided_dgrad");
    else if (KS)
      snprintf(buf, sizeof buf, "%s<%s,%d,%d,%d,%d,%s,%d,%d>", base, tname<T>(), BM, BN, WM, WN,
               FLAT ? "true" : "false", KS, PF);
    else
      snprintf(buf, sizeof buf, "%s<%s,%d,%d,%d,%d,%s>", base, tname<T>(), BM, BN, WM, WN,
               FLAT ? "true" : "false");
    init = true;
  }
  return buf;
}

template <typename T, int BM, int BN, int WM, int WN, int KS, int PF = 1, int GM = 0>
static hipError_t conv_go(const ConvArgs& a, bool flat, hipStream_t s, int* grid_rows = nullptr) {
  static_assert(GM >= 0 && GM <= 2, "gather mode");
  int M = a.nb * (GM ? a.Ho * a.Wo : a.H * a.W);
  dim3 grid((M + BM - 1) / BM, (a.N + BN - 1) / BN);
  if (grid_rows) *grid_rows = (int)grid.x;
  // algorithmic work: every (row, tap) pair of the convolution once; a strided
  // data gradient reads each output-gradient pixel once per tap
  double flops = 2.0 * a.nb * (GM == 2 ? a.H * a.W : M / a.nb) * (double)a.N * a.R * a.S * a.C;
  if (flat)
    XP_LAUNCH((kname<T, BM, BN, WM, WN, true, KS, PF, GM>("k_conv_gemm")), flops,
              (k_conv_gemm<T, BM, BN, WM, WN, true, KS, PF, GM>), grid, dim3(WM * WN * 64), 0, s, a);
  else
    XP_LAUNCH((kname<T, BM, BN, WM, WN, false, KS, PF, GM>("k_conv_gemm")), flops,
              (k_conv_gemm<T, BM, BN, WM, WN, false, KS, PF, GM>), grid, dim3(WM * WN * 64), 0, s, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t conv_dispatch(const ConvArgs& a0, hipStream_t s, int* gr) {
  constexpr int VEC = MT<T>::VEC;
  ConvArgs a = a0;
  if (a.stride < 1) a.stride = 1;
  const size_t M = (size_t)a.nb * a.H * a.W;
  // the 16-byte chunk path addresses both operands with 32-bit buffer offsets
  const bool spans = ((M - 1) * a.ldx + a.C) * sizeof(T) < ((size_t)1 << 31) &&
                     (size_t)a.N * a.R * a.S * a.C * sizeof(T) < ((size_t)1 << 31);
  bool flat = (a.C % VEC) != 0 || (a.ldx % VEC) != 0 ||
              (reinterpret_cast<uintptr_t>(a.x) % 16) != 0 ||
              (reinterpret_cast<uintptr_t>(a.w) % 16) != 0 || !spans;
  const bool narrow = a.N <= 32;
  if (a.tr || a.Ho > 0) {
    // strided or unpadded layers (ResNet-101 stem, first blocks, projections;
    // Inception-V3 stem and grid reductions): general tiles
    if constexpr (sizeof(T) == 2) {
      // large grids (first stages at 224 x 224 over micro-batch 100): 128-row
      // tiles, or one 96-column tile for 64 < N <= 96; 10-33% faster there
      const size_t rows = (size_t)a.nb * a.Ho * a.Wo;
      if (!flat && !narrow && rows >= 65536) {
        if (a.tr) {
          if (a.N <= 64) return conv_go<T, 128, 64, 2, 2, 2, 2, 2>(a, flat, s, gr);
          if (a.N <= 96) return conv_go<T, 64, 96, 2, 2, 1, 2, 2>(a, flat, s, gr);
          return conv_go<T, 128, 128, 2, 4, 2, 2, 2>(a, flat, s, gr);
        }
        if (a.N <= 64) return conv_go<T, 128, 64, 2, 2, 2, 2, 1>(a, flat, s, gr);
        if (a.N <= 96) return conv_go<T, 64, 96, 2, 2, 1, 2, 1>(a, flat, s, gr);
        return conv_go<T, 128, 128, 2, 4, 2, 2, 1>(a, flat, s, gr);
      }
      if (a.tr) {
        if (narrow) return conv_go<T, 64, 32, 2, 2, 1, 2, 2>(a, flat, s, gr);
        return conv_go<T, 64, 64, 2, 2, 2, 2, 2>(a, flat, s, gr);
      }
      if (narrow) return conv_go<T, 64, 32, 2, 2, 1, 2, 1>(a, flat, s, gr);
      return conv_go<T, 64, 64, 2, 2, 2, 2, 1>(a, flat, s, gr);
    } else {
      if (a.tr) {
        if (narrow) return conv_go<T, 64, 32, 2, 2, 1, 1, 2>(a, flat, s, gr);
        return conv_go<T, 64, 64, 2, 2, 1, 1, 2>(a, flat, s, gr);
      }
      if (narrow) return conv_go<T, 64, 32, 2, 2, 1, 1, 1>(a, flat, s, gr);
      return conv_go<T, 64, 64, 2, 2, 1, 1, 1>(a, flat, s, gr);
    }
  }
  if constexpr (sizeof(T) == 2) {
    // From a sweep of the stage shapes on MI355X (tile, stage depth KS,
    // register prefetch depth PF)
    const int taps = a.R * a.S;
    const int ks = flat ? 1 : pick_ks_bf16(a.C, taps);
    // KS counts 32-deep slices for the 16x16 MFMA tiles and 16-deep slices
    // for the 32x32 ones (64x64 on 2x2 waves), so 64x64 KS 2 has BK = 32.
    if (narrow) {
      if (ks == 4) return conv_go<T, 32, 32, 2, 2, 4, 3>(a, flat, s, gr);
      if (ks == 2) return conv_go<T, 32, 32, 2, 2, 2, 3>(a, flat, s, gr);
      return conv_go<T, 64, 32, 2, 2, 1, 2>(a, flat, s, gr);
    }
    // large images (ResNet-101 at 224 x 224 over micro-batch 100: 78 400 to
    // 313 600 rows): 128-row tiles, 128 columns on eight waves where N allows;
    // 4-17% faster there than the 32- and 64-row tiles
    if (!flat && M >= 65536 && (a.N <= 64 || a.N >= 128)) {
      if (a.N <= 64) return conv_go<T, 128, 64, 2, 2, 2, 2>(a, flat, s, gr);
      return conv_go<T, 128, 128, 2, 4, 2, 2>(a, flat, s, gr);
    }
    // one 96-column tile reads the input once and wastes no MFMA columns
    if (!flat && taps > 1 && taps < 25 && a.N > 64 && a.N <= 96)
      return conv_go<T, 64, 96, 2, 2, 1, 2>(a, flat, s, gr);
    if (ks == 1) return conv_go<T, 64, 64, 2, 2, 2, 2>(a, flat, s, gr);
    if (!flat && taps == 1 && a.N > 96 && M >= 16384) {
      // wide 1x1 (merged siblings) over many rows: 64-row tiles, the column
      // tile that pads N least
      if ((a.N + 95) / 96 * 96 <= (a.N + 63) / 64 * 64)
        return conv_go<T, 64, 96, 2, 2, 1, 2>(a, flat, s, gr);
      return conv_go<T, 64, 64, 2, 2, 2, 2>(a, flat, s, gr);
    }
    if (taps >= 25 && a.N > 48) {
      if (ks == 4) return conv_go<T, 64, 64, 2, 2, 8, 2>(a, flat, s, gr);
      return conv_go<T, 64, 64, 2, 2, 4, 2>(a, flat, s, gr);
    }
    if (ks == 4) return conv_go<T, 32, 64, 2, 2, 4, 2>(a, flat, s, gr);
    return conv_go<T, 32, 64, 2, 2, 2, 2>(a, flat, s, gr);
  } else {
    if (narrow) return conv_go<T, 64, 32, 2, 2, 1>(a, flat, s, gr);
    return conv_go<T, 64, 64, 2, 2, 1>(a, flat, s, gr);
  }
}

hipError_t launch_conv_gemm(int dtype, const ConvArgs& a, hipStream_t s, int* grid_rows) {
  if (grid_rows) *grid_rows = 0;
  if (a.nb * a.H * a.W <= 0 || a.N <= 0) return hipSuccess;
  return dtype == DT_BF16 ? conv_dispatch<bf16_t>(a, s, grid_rows)
                          : conv_dispatch<float>(a, s, grid_rows);
}

int conv_max_row_tiles(int M) { return (M + 31) / 32; }

// The weight gradient of a filter with 65..96 output channels and K >= 768
// takes one 96 x 128 tile per K block (all output channels at once, the
// 32x32x16 form): 3x3 96 -> 96 over 32 x 35 x 35 pixels, 35.9 -> 31.1 us
// with its split reduction
static bool wgrad_tile96(int N, int K, int taps) { return N > 64 && N <= 96 && taps > 1 && K >= 768; }
// A 1x1 filter with 129..192 output channels (the merged 1x1 siblings of an
// Inception-A module: 176) takes one 192 x 64 tile per K block, about 256
// workgroups: 256 -> 176 over 32 x 35 x 35 pixels, 28.6 -> 22.5 us with its
// split reduction
static bool wgrad_tile192(int N, int taps) { return N > 128 && N <= 192 && taps == 1; }

int wgrad_pick_splits(int dtype, int M, int N, int K, int taps) {
  // bf16: 64x64 tiles, about 512 workgroups (1x1) or 1024 (larger filters),
  // from a sweep of the stage shapes; fp32/fp64: the tile of wgrad_dispatch
  // and about 512 workgroups
  const bool bf = dtype == DT_BF16;
  // bf16, 65..96 output channels of a filter with K >= 768: one 96-row tile
  // by 128 columns (k_wgrad_t<96,128>), about 512 workgroups
  const bool t96 = bf && wgrad_tile96(N, K, taps);
  const bool t192 = bf && !t96 && wgrad_tile192(N, taps);
  int bm = t96 ? 96 : t192 ? 192 : bf ? 64 : (N <= 64 ? 64 : 128);
  int bn = t96 ? 128 : bf ? 64 : (K <= 64 ? 64 : 128);
  int tiles = ((N + bm - 1) / bm) * ((K + bn - 1) / bn);
  // enough tiles to fill the chip: one split, added straight into the
  // accumulator (VGG-16's 512 x 4608 gradients at 8 x 8: 72.9 -> 61.5 us)
  if (bf && tiles >= 512) return 1;
  int target = t96 ? 512 : t192 ? 256 : bf && taps > 1 ? 1024 : 512;
  int want = (target + tiles - 1) / tiles;
  // at least ~128 pixels per split (VGG-16's 3-channel first layer, one tile:
  // 128 -> 256 splits, 28 -> 20 us with the reduction)
  int maxs = (M + 127) / 128;
  // keep the partial sums (written and read back once) below the operands' bytes
  int64_t op_bytes = (int64_t)M * (N + K / 1) * 2;
  int64_t part_bytes = (int64_t)N * K * 4;
  int64_t maxb = part_bytes > 0 ? op_bytes / part_bytes : want;
  if (maxb < 4) maxb = 4;
  if (want > maxs) want = maxs;
  if (want > maxb) want = (int)maxb;
  if (want < 1) want = 1;
  return want;
}
size_t wgrad_part_bytes(int dtype, int N, int K, int splits) {
  return (size_t)splits * N * K * (dtype == DT_BF16 ? sizeof(float) : sizeof(double));
}

// grad (+)= the fixed-order sum of the launch's split partials
template <typename T>
static hipError_t wgrad_reduce(const WgradArgs& a, hipStream_t s) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int K = a.R * a.S * a.C;
  int64_t count = (int64_t)a.N * K;
  int blocks = (int)(((count + 3) / 4 + (256 / SPLIT_GROUPS) - 1) / (256 / SPLIT_GROUPS));
  typedef typename MT<T>::part_t P;
  GradDst d{};
  if (a.nseg > 0) {
    d.nseg = a.nseg;
    for (int j = 0; j <= a.nseg; ++j) d.base[j] = (int64_t)a.seg_row0[j] * K;
    for (int j = 0; j < a.nseg; ++j) d.ptr[j] = a.seg_grad[j];
  } else {
    d.nseg = 1;
    d.base[0] = 0;
    d.base[1] = count;
    d.ptr[0] = a.grad;
  }
  XP_LAUNCH(sizeof(P) == 4 ? "k_split_reduce<float>" : "k_split_reduce<double>",
            (double)count * (a.splits * sizeof(P) + 8), k_split_reduce<P>, dim3(blocks), dim3(256), 0, s,
            (const P*)a.part, a.splits, count, d);
  return hipGetLastError();
}

template <typename T, int BM, int BN, int WM, int WN>
static hipError_t wgrad_go(const WgradArgs& a, bool flat, hipStream_t s) {
  int K = a.R * a.S * a.C;
  dim3 grid((a.N + BM - 1) / BM, (K + BN - 1) / BN, a.splits);
  const int pix = a.Ho > 0 ? a.Ho * a.Wo : a.H * a.W;
  double flops = 2.0 * a.nb * pix * (double)a.N * K;
  if (flat)
    XP_LAUNCH((kname<T, BM, BN, WM, WN, true>("k_wgrad")), flops, (k_wgrad<T, BM, BN, WM, WN, true>),
              grid, dim3(256), 0, s, a);
  else
    XP_LAUNCH((kname<T, BM, BN, WM, WN, false>("k_wgrad")), flops, (k_wgrad<T, BM, BN, WM, WN, false>),
              grid, dim3(256), 0, s, a);
  return wgrad_reduce<T>(a, s);
}

template <int BM, int BN, int WM, int WN, int PF, bool GRID = false>
static hipError_t wgrad_t_go(const WgradArgs& a, hipStream_t s) {
  int K = a.R * a.S * a.C;
  dim3 grid((a.N + BM - 1) / BM, (K + BN - 1) / BN, a.splits);
  const int pix = a.Ho > 0 ? a.Ho * a.Wo : a.H * a.W;
  double flops = 2.0 * a.nb * pix * (double)a.N * K;
  static char name[64];
  snprintf(name, sizeof name, GRID ? "k_wgrad_t<%d,%d,%d,%d,%d,grid>" : "k_wgrad_t<%d,%d,%d,%d,%d>", BM, BN,
           WM, WN, PF);
  WgradArgs b = a;
  b.direct = a.splits == 1;
  XP_LAUNCH(name, flops, (k_wgrad_t<BM, BN, WM, WN, PF, GRID>), grid, dim3(256), 0, s, b);
  if (b.direct) return hipGetLastError();
  return wgrad_reduce<bf16_t>(a, s);
}


template <typename T>
static hipError_t wgrad_dispatch(const WgradArgs& a, hipStream_t s) {
  constexpr int VEC = MT<T>::VEC;
  bool flat = (a.C % VEC) != 0 || (a.ldx % VEC) != 0 ||
              (reinterpret_cast<uintptr_t>(a.x) % 16) != 0;
  int K = a.R * a.S * a.C;
  bool n64 = a.N <= 64, k64 = K <= 64;
  if constexpr (sizeof(T) == 2) {
    const int M = a.nb * (a.Ho > 0 ? a.Ho * a.Wo : a.H * a.W), Min = a.nb * a.H * a.W;
    const bool chunks = !flat && (a.N % VEC) == 0 && (a.lddz % VEC) == 0 &&
                        (reinterpret_cast<uintptr_t>(a.dz) % 16) == 0 &&
                        (((size_t)(M - 1)) * a.lddz + a.N) * sizeof(T) < ((size_t)1 << 31) &&
                        (((size_t)(Min - 1)) * a.ldx + a.C) * sizeof(T) < ((size_t)1 << 31);
    // same grid and square padding: pixel offsets shift with the pixel index;
    // otherwise each pixel addresses x from its own row and column
    if (chunks && a.Ho <= 0 && a.pad == a.padw && wgrad_tile96(a.N, K, a.R * a.S))
      return wgrad_t_go<96, 128, 1, 4, 2>(a, s);
    if (chunks && a.Ho <= 0 && a.pad == a.padw && wgrad_tile192(a.N, a.R * a.S))
      return wgrad_t_go<192, 64, 2, 2, 1>(a, s);
    if (chunks && a.Ho <= 0 && a.pad == a.padw) return wgrad_t_go<64, 64, 2, 2, 1>(a, s);
    if (chunks) return wgrad_t_go<64, 64, 2, 2, 1, true>(a, s);
  }
  if (n64 && k64) return wgrad_go<T, 64, 64, 2, 2>(a, flat, s);
  if (n64) return wgrad_go<T, 64, 128, 2, 2>(a, flat, s);
  if (k64) return wgrad_go<T, 128, 64, 2, 2>(a, flat, s);
  return wgrad_go<T, 128, 128, 2, 2>(a, flat, s);
}

hipError_t launch_wgrad(int dtype, const WgradArgs& a, hipStream_t s) {
  if (a.N <= 0) return hipSuccess;
  return dtype == DT_BF16 ? wgrad_dispatch<bf16_t>(a, s) : wgrad_dispatch<float>(a, s);
}

hipError_t launch_gather(int dtype, const GatherArgs& a, hipStream_t s) {
  if (a.nseg < 0 || a.nseg > GATHER_BATCH) return hipErrorInvalidValue;
  int64_t total = 0, longest = 0;
  for (int j = 0; j < a.nseg; ++j) {
    total += a.count[j];
    longest = a.count[j] > longest ? a.count[j] : longest;
  }
  if (total <= 0) return hipSuccess;
  int blocks = (int)((longest + 255) / 256);
  if (blocks > 1024) blocks = 1024;
  if (dtype == DT_BF16)
    XP_LAUNCH("k_gather<bf16>", (double)total * 4, k_gather<bf16_t>, dim3(blocks), dim3(256), 0, s, a);
  else
    XP_LAUNCH("k_gather<f32>", (double)total * 8, k_gather<float>, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_flip_set(int dtype, const FlipSet& f, hipStream_t s) {
  if (f.n <= 0) return hipSuccess;
  if (f.n > FLIP_MAX) return hipErrorInvalidValue;
  int64_t most = 0, total = 0;
  for (int q = 0; q < f.n; ++q) {
    const int64_t e = (int64_t)f.N[q] * f.R[q] * f.S[q] * f.C[q];
    most = std::max(most, e);
    total += e;
  }
  if (most <= 0) return hipSuccess;
  int blocks = (int)((most + 255) / 256);
  if (blocks > 1024) blocks = 1024;
  if (dtype == DT_BF16)
    XP_LAUNCH("k_flip_set<bf16>", (double)total * 4, k_flip_set<bf16_t>, dim3(blocks, f.n), dim3(256), 0, s, f);
  else
    XP_LAUNCH("k_flip_set<f32>", (double)total * 8, k_flip_set<float>, dim3(blocks, f.n), dim3(256), 0, s, f);
  return hipGetLastError();
}


}  // namespace xp
