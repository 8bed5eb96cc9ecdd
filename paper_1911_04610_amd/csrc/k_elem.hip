// Memory-bound layer kernels: batch-norm statistics and backward reductions,
// fused BN (+ residual add) (+ ReLU) apply, element-wise ReLU / add / mask,
// max / average pooling, global average pooling and softmax cross-entropy.
//
// Activations are NHWC views (row = pixel, column = channel).  Kernels that
// walk a view put 64 consecutive channels on the lanes of a wave (coalesced
// row segments) and spread rows over the 4 waves of a workgroup and over
// blockIdx.y.  Arithmetic is fp64; every stored value is rounded once.
// Reductions are two-level with a fixed order (per-block partials, then one
// thread per column), so results do not depend on scheduling.
#include "xp_device.h"
#include "xp_kernels.h"

#include <algorithm>
#include <initializer_list>
#include <utility>

namespace xp {

__host__ __device__ static inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

static int row_blocks_for(int M, int C) {
  int chunks = ceil_div(C, 64);
  int want = ceil_div(1024, chunks);            // about 1024 workgroups in total
  int maxrb = ceil_div(M, 64);                  // at least ~64 rows per workgroup
  if (want > maxrb) want = maxrb;
  if (want < 1) want = 1;
  return want;
}

int col_row_blocks(int M, int C) { return row_blocks_for(M, C); }
int col_row_blocks_v(int M, int C, int N);
// the vectorised reduction uses at most this many row blocks
constexpr int COL_MAX_ROW_BLOCKS_V = 1024;
size_t col_partial_bytes(int M, int C) {
  int rb = row_blocks_for(M, C);
  if (rb < COL_MAX_ROW_BLOCKS_V) rb = COL_MAX_ROW_BLOCKS_V;
  return (size_t)rb * 2 * C * sizeof(double);
}

// ---------------------------------------------------------------- column reductions
template <typename T>
__global__ __launch_bounds__(256) void k_colpart(ColArgs a) {
  __shared__ double sh[2][4][64];
  const int lanec = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lanec;
  const int per = ceil_div(a.M, a.row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(a.M, r0 + per);
  const T* A = (const T*)a.a;
  const T* Z = (const T*)a.z;
  double s0 = 0.0, s1 = 0.0;
  if (col < a.C) {
    if (a.mode == COL_STATS) {
      for (int r = r0 + rg; r < r1; r += 4) {
        double v = ldd(A + (size_t)r * a.lda + col);
        s0 += v;
        s1 += v * v;
      }
    } else if (a.mode == COL_BNBWD) {
      const double mu = a.mean[col], rs = a.rstd[col];
      for (int r = r0 + rg; r < r1; r += 4) {
        double g = ldd(A + (size_t)r * a.lda + col);
        double xh = (ldd(Z + (size_t)r * a.ldz + col) - mu) * rs;
        s0 += g;
        s1 += g * xh;
      }
    } else {
      for (int r = r0 + rg; r < r1; r += 4) s0 += ldd(A + (size_t)r * a.lda + col);
    }
  }
  sh[0][rg][lanec] = s0;
  sh[1][rg][lanec] = s1;
  __syncthreads();
  if (rg == 0 && col < a.C) {
    double t0 = ((sh[0][0][lanec] + sh[0][1][lanec]) + sh[0][2][lanec]) + sh[0][3][lanec];
    double t1 = ((sh[1][0][lanec] + sh[1][1][lanec]) + sh[1][2][lanec]) + sh[1][3][lanec];
    a.partial[((size_t)col * 2 + 0) * a.row_blocks + blockIdx.y] = t0;
    a.partial[((size_t)col * 2 + 1) * a.row_blocks + blockIdx.y] = t1;
  }
}

hipError_t launch_colfinal(const ColArgs& a, hipStream_t s);

template <typename T>
static hipError_t colreduce_go(const ColArgs& a, hipStream_t s) {
  dim3 grid(ceil_div(a.C, 64), a.row_blocks);
  XP_LAUNCH(sizeof(T) == 2 ? "k_colpart<bf16>" : "k_colpart<f32>", (double)a.M * a.C * sizeof(T) * (a.mode == COL_BNBWD ? 2 : 1), k_colpart<T>, grid,
            dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_colfinal(a, s);
}

static hipError_t launch_colreduce_s(int dtype, const ColArgs& a, hipStream_t s) {
  if (a.C <= 0) return hipSuccess;
  return dtype == DT_BF16 ? colreduce_go<bf16_t>(a, s) : colreduce_go<float>(a, s);
}

// ---------------------------------------------------------------- BN apply / backward
template <typename T>
__global__ __launch_bounds__(256) void k_bn_apply(BnApplyArgs a, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int per = ceil_div(a.M, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(a.M, r0 + per);
  const double mu = a.mean[col], rs = a.rstd[col];
  const double g = (double)a.gamma[col], b = (double)a.beta[col];
  const T* Z = (const T*)a.z;
  const T* R = (const T*)a.res;
  T* Y = (T*)a.y;
  for (int r = r0 + rg; r < r1; r += 4) {
    double xh = (ldd(Z + (size_t)r * a.ldz + col) - mu) * rs;
    double v = g * xh + b;
    // a BN output is a layer output of its own: rounded to the storage type
    // before the residual add takes it in (the sum is rounded on store)
    if (R) v = rnd<T>(v) + ldd(R + (size_t)r * a.ldres + col);
    if (a.relu) v = v > 0.0 ? v : 0.0;
    std_(Y + (size_t)r * a.ldy + col, v);
  }
}

static hipError_t launch_bn_apply_s(int dtype, const BnApplyArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    XP_LAUNCH("k_bn_apply<bf16>", (double)a.M * a.C * 2 * (a.res ? 3 : 2), k_bn_apply<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    XP_LAUNCH("k_bn_apply<f32>", (double)a.M * a.C * 4 * (a.res ? 3 : 2), k_bn_apply<float>, grid, dim3(256), 0, s, a, rb);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_bn_bwd(BnBwdArgs a, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int per = ceil_div(a.M, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(a.M, r0 + per);
  const double mu = a.mean[col], rs = a.rstd[col];
  const double gam = (double)a.gamma[col];
  const double db_M = a.dbeta[col] / a.M, dg_M = a.dgamma[col] / a.M;
  const T* G = (const T*)a.g;
  const T* Z = (const T*)a.z;
  T* DZ = (T*)a.dz;
  T* DR = (T*)a.dres;
  const T* RM = (const T*)a.resmask;
  const T* ZM = (const T*)a.dzmask;
  for (int r = r0 + rg; r < r1; r += 4) {
    double g = ldd(G + (size_t)r * a.ldg + col);
    double xh = (ldd(Z + (size_t)r * a.ldz + col) - mu) * rs;
    double dzv = gam * rs * (g - db_M - xh * dg_M);
    if (ZM && !(ldd(ZM + (size_t)r * a.ldzm + col) > 0.0)) dzv = 0.0;
    T* pz = DZ + (size_t)r * a.lddz + col;
    if (a.dz_accumulate) dzv += ldd(pz);
    std_(pz, dzv);
    if (DR) {
      double d = g;
      if (RM && !(ldd(RM + (size_t)r * a.ldrm + col) > 0.0)) d = 0.0;
      T* p = DR + (size_t)r * a.lddres + col;
      if (a.res_accumulate) d += ldd(p);
      std_(p, d);
    }
  }
}

static hipError_t launch_bn_bwd_s(int dtype, const BnBwdArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    XP_LAUNCH("k_bn_bwd<bf16>", (double)a.M * a.C * 2 * (a.dres ? 5 : 3), k_bn_bwd<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    XP_LAUNCH("k_bn_bwd<f32>", (double)a.M * a.C * 4 * (a.dres ? 5 : 3), k_bn_bwd<float>, grid, dim3(256), 0, s, a, rb);
  return hipGetLastError();
}

// ---------------------------------------------------------------- element-wise
template <typename T>
__global__ __launch_bounds__(256) void k_elt(EltArgs a, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int per = ceil_div(a.M, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(a.M, r0 + per);
  const T* A = (const T*)a.a;
  const T* B = (const T*)a.b;
  const T* MK = (const T*)a.mask;
  T* Y = (T*)a.y;
  for (int r = r0 + rg; r < r1; r += 4) {
    double v = ldd(A + (size_t)r * a.lda + col);
    if (B) v += ldd(B + (size_t)r * a.ldb + col);
    if (a.relu) v = v > 0.0 ? v : 0.0;
    if (MK && !(ldd(MK + (size_t)r * a.ldm + col) > 0.0)) v = 0.0;
    T* p = Y + (size_t)r * a.ldy + col;
    if (a.accumulate) v += ldd(p);
    std_(p, v);
  }
}

static hipError_t launch_elementwise_s(int dtype, const EltArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    XP_LAUNCH("k_elt<bf16>", (double)a.M * a.C * 2 * 3, k_elt<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    XP_LAUNCH("k_elt<f32>", (double)a.M * a.C * 4 * 3, k_elt<float>, grid, dim3(256), 0, s, a, rb);
  return hipGetLastError();
}

// ---------------------------------------------------------------- pooling
// rows of the launch grid walk output pixels (forward) or input pixels (backward)
template <typename T>
__global__ __launch_bounds__(256) void k_maxpool_fwd(PoolArgs a, int rows, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int Ho = a.H / 2, Wo = a.W / 2;
  const int per = ceil_div(rows, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(rows, r0 + per);
  const T* X = (const T*)a.x;
  T* O = (T*)a.out;
  for (int r = r0 + rg; r < r1; r += 4) {
    int n = r / (Ho * Wo), rem = r - n * Ho * Wo, ho = rem / Wo, wo = rem - ho * Wo;
    const T* base = X + ((size_t)(n * a.H + 2 * ho) * a.W + 2 * wo) * a.ldx + col;
    T best = base[0];
    double bv = ldd(&best);
    const T cand[3] = {base[a.ldx], base[(size_t)a.W * a.ldx], base[((size_t)a.W + 1) * a.ldx]};
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      double cv = ldd(&cand[q]);
      if (cv > bv) { bv = cv; best = cand[q]; }
    }
    O[(size_t)r * a.ldo + col] = best;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_maxpool_bwd(PoolArgs a, int rows, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int Ho = a.H / 2, Wo = a.W / 2;
  const int per = ceil_div(rows, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(rows, r0 + per);
  const T* X = (const T*)a.x;
  const T* DY = (const T*)a.dy;
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  for (int r = r0 + rg; r < r1; r += 4) {
    int n = r / (a.H * a.W), rem = r - n * a.H * a.W, h = rem / a.W, w = rem - h * a.W;
    double d = 0.0;
    int ho = h >> 1, wo = w >> 1;
    if (ho < Ho && wo < Wo) {
      const T* base = X + ((size_t)(n * a.H + 2 * ho) * a.W + 2 * wo) * a.ldx + col;
      double v[4] = {ldd(base), ldd(base + a.ldx), ldd(base + (size_t)a.W * a.ldx),
                     ldd(base + ((size_t)a.W + 1) * a.ldx)};
      int arg = 0;
#pragma unroll
      for (int q = 1; q < 4; ++q)
        if (v[q] > v[arg]) arg = q;  // first maximum in row-major order wins ties
      if (arg == ((h & 1) << 1) + (w & 1))
        d = ldd(DY + ((size_t)(n * Ho + ho) * Wo + wo) * a.lddy + col);
    }
    if (MK && !(ldd(MK + (size_t)r * a.ldm + col) > 0.0)) d = 0.0;
    T* p = O + (size_t)r * a.ldo + col;
    if (a.accumulate) d += ldd(p);
    std_(p, d);
  }
}

// 3x3 / stride 1 / pad 1 / divisor 9.  The window is symmetric and the divisor
// constant, so the backward is the same stencil applied to the output gradient.
template <typename T>
__global__ __launch_bounds__(256) void k_avgpool3(PoolArgs a, const T* src, int ld_src,
                                                   int rows, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int per = ceil_div(rows, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(rows, r0 + per);
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  for (int r = r0 + rg; r < r1; r += 4) {
    int n = r / (a.H * a.W), rem = r - n * a.H * a.W, h = rem / a.W, w = rem - h * a.W;
    double sum = 0.0;
#pragma unroll
    for (int dr = -1; dr <= 1; ++dr)
#pragma unroll
      for (int ds = -1; ds <= 1; ++ds) {
        int hh = h + dr, ww = w + ds;
        if (hh >= 0 && hh < a.H && ww >= 0 && ww < a.W)
          sum += ldd(src + ((size_t)(n * a.H + hh) * a.W + ww) * ld_src + col);
      }
    double v = sum / 9.0;
    if (MK && !(ldd(MK + (size_t)r * a.ldm + col) > 0.0)) v = 0.0;
    T* p = O + (size_t)r * a.ldo + col;
    if (a.accumulate) v += ldd(p);
    std_(p, v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_gap_fwd(PoolArgs a) {
  __shared__ double sh[4][64];
  const int lanec = threadIdx.x & 63, rg = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lanec, n = blockIdx.y;
  const int HW = a.H * a.W;
  const T* X = (const T*)a.x;
  double s = 0.0;
  if (col < a.C)
    for (int p = rg; p < HW; p += 4) s += ldd(X + ((size_t)n * HW + p) * a.ldx + col);
  sh[rg][lanec] = s;
  __syncthreads();
  if (rg == 0 && col < a.C) {
    double t = ((sh[0][lanec] + sh[1][lanec]) + sh[2][lanec]) + sh[3][lanec];
    std_((T*)a.out + (size_t)n * a.ldo + col, t / HW);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_gap_bwd(PoolArgs a, int rows, int row_blocks) {
  const int col = blockIdx.x * 64 + (threadIdx.x & 63), rg = threadIdx.x >> 6;
  if (col >= a.C) return;
  const int HW = a.H * a.W;
  const int per = ceil_div(rows, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(rows, r0 + per);
  const T* DY = (const T*)a.dy;
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  for (int r = r0 + rg; r < r1; r += 4) {
    int n = r / HW;
    double d = ldd(DY + (size_t)n * a.lddy + col) / HW;
    if (MK && !(ldd(MK + (size_t)r * a.ldm + col) > 0.0)) d = 0.0;
    T* p = O + (size_t)r * a.ldo + col;
    if (a.accumulate) d += ldd(p);
    std_(p, d);
  }
}

template <typename T>
static void pool_launch_rows(void (*k)(PoolArgs, int, int), const char* name, const PoolArgs& a,
                             int rows, hipStream_t s) {
  int rb = row_blocks_for(rows, a.C);
  XP_LAUNCH(name, (double)rows * a.C * sizeof(T) * 3, k, dim3(ceil_div(a.C, 64), rb), dim3(256), 0, s, a, rows, rb);
}

static hipError_t launch_maxpool_fwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * (a.H / 2) * (a.W / 2);
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_maxpool_fwd<bf16_t>, "k_maxpool_fwd<bf16>", a, rows, s);
  else pool_launch_rows<float>(k_maxpool_fwd<float>, "k_maxpool_fwd<f32>", a, rows, s);
  return hipGetLastError();
}

static hipError_t launch_maxpool_bwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_maxpool_bwd<bf16_t>, "k_maxpool_bwd<bf16>", a, rows, s);
  else pool_launch_rows<float>(k_maxpool_bwd<float>, "k_maxpool_bwd<f32>", a, rows, s);
  return hipGetLastError();
}

template <typename T>
static hipError_t avg_go(const PoolArgs& a, const void* src, int ld_src, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(rows, a.C);
  XP_LAUNCH("k_avgpool3", (double)rows * a.C * sizeof(T) * 2, k_avgpool3<T>, dim3(ceil_div(a.C, 64), rb), dim3(256), 0, s, a,
                     (const T*)src, ld_src, rows, rb);
  return hipGetLastError();
}

static hipError_t launch_avgpool_fwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  return dtype == DT_BF16 ? avg_go<bf16_t>(a, a.x, a.ldx, s) : avg_go<float>(a, a.x, a.ldx, s);
}

static hipError_t launch_avgpool_bwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  return dtype == DT_BF16 ? avg_go<bf16_t>(a, a.dy, a.lddy, s) : avg_go<float>(a, a.dy, a.lddy, s);
}

static hipError_t launch_gap_fwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  if (a.nb <= 0 || a.C <= 0) return hipSuccess;
  dim3 grid(ceil_div(a.C, 64), a.nb);
  double gb = (double)a.nb * a.H * a.W * a.C * (dtype == DT_BF16 ? 2 : 4);
  if (dtype == DT_BF16) XP_LAUNCH("k_gap_fwd<bf16>", gb, k_gap_fwd<bf16_t>, grid, dim3(256), 0, s, a);
  else XP_LAUNCH("k_gap_fwd<f32>", gb, k_gap_fwd<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

static hipError_t launch_gap_bwd_s(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_gap_bwd<bf16_t>, "k_gap_bwd<bf16>", a, rows, s);
  else pool_launch_rows<float>(k_gap_bwd<float>, "k_gap_bwd<f32>", a, rows, s);
  return hipGetLastError();
}

// ============================================================================
// vectorised forms: each thread moves 16-byte chunks (8 bf16 or 4 fp32
// channels).  Used whenever channel counts, row pitches and base pointers
// allow 16-byte accesses (every layer of the stages measured here); the
// per-channel kernels above remain for the other shapes.
// ============================================================================
template <typename T> struct VT;
template <> struct VT<bf16_t> { static constexpr int N = 8; };
template <> struct VT<float> { static constexpr int N = 4; };

// a 16-byte chunk as raw bits, and its values widened to double
template <typename T>
XP_DEV uint4 ld16(const T* p) { return *reinterpret_cast<const uint4*>(p); }
template <typename T>
XP_DEV void cvt16(uint4 u, double* v);
template <>
XP_DEV void cvt16<bf16_t>(uint4 u, double* v) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = (double)__uint_as_float(w[i] << 16);
    v[2 * i + 1] = (double)__uint_as_float(w[i] & 0xffff0000u);
  }
}
template <>
XP_DEV void cvt16<float>(uint4 u, double* v) {
  v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y);
  v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
}
template <typename T>
XP_DEV void vld(const T* p, double* v) { cvt16<T>(ld16(p), v); }
// a chunk of values rounded to the storage type, as raw bits
template <typename T>
XP_DEV uint4 pack16(const double* v);
template <>
XP_DEV uint4 pack16<bf16_t>(const double* v) {
  uint4 u;
  u.x = f32x2_to_bf16x2((float)v[0], (float)v[1]);
  u.y = f32x2_to_bf16x2((float)v[2], (float)v[3]);
  u.z = f32x2_to_bf16x2((float)v[4], (float)v[5]);
  u.w = f32x2_to_bf16x2((float)v[6], (float)v[7]);
  return u;
}
template <>
XP_DEV uint4 pack16<float>(const double* v) {
  return make_uint4(__float_as_uint((float)v[0]), __float_as_uint((float)v[1]),
                    __float_as_uint((float)v[2]), __float_as_uint((float)v[3]));
}
template <typename T>
XP_DEV void vst(T* p, const double* v) { *reinterpret_cast<uint4*>(p) = pack16<T>(v); }

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <typename T>
static bool vec_ok(int C, std::initializer_list<std::pair<const void*, int>> views) {
  constexpr int N = VT<T>::N;
  if (C % N) return false;
  for (auto& v : views)
    if (v.first && (!al16(v.first) || (v.second % N))) return false;
  return true;
}

static int grid_for(int64_t items) {
  int64_t b = (items + 255) / 256;
  if (b > 8192) b = 8192;
  return (int)(b < 1 ? 1 : b);
}

// mask helper: zero lanes whose mask value is not > 0
template <typename T>
XP_DEV void vmask_raw(uint4 mk, double* v) {
  constexpr int N = VT<T>::N;
  double m[N];
  cvt16<T>(mk, m);
#pragma unroll
  for (int e = 0; e < N; ++e)
    if (!(m[e] > 0.0)) v[e] = 0.0;
}
template <typename T>
XP_DEV void vmask(const T* mk, double* v) { vmask_raw<T>(ld16(mk), v); }

// Row kernels (BN apply / backward): a block holds CPB chunk columns x RPB
// row lanes, each thread keeps its chunk's per-channel coefficients in
// registers and walks rows with a grid-wide stride, U rows per trip, every
// load of a trip issued before its arithmetic.
struct RowMap {
  int chunk, row0, stride;
  bool live;
};
template <typename T>
XP_DEV RowMap row_map(int C) {
  constexpr int N = VT<T>::N;
  const int chunks = C / N;
  const int cpb = chunks < 256 ? chunks : 256;
  const int rpb = 256 / cpb;
  const int rl = threadIdx.x / cpb;
  RowMap m;
  m.chunk = blockIdx.y * cpb + (int)(threadIdx.x % cpb);
  m.live = rl < rpb && m.chunk < chunks;
  m.row0 = blockIdx.x * rpb + rl;
  m.stride = gridDim.x * rpb;
  return m;
}
// grid of a row kernel: about U rows per thread
static dim3 row_grid(int64_t M, int C, int N, int U) {
  const int chunks = C / N;
  const int cpb = chunks < 256 ? chunks : 256;
  const int rpb = 256 / cpb;
  int64_t gx = (M + (int64_t)rpb * U - 1) / ((int64_t)rpb * U);
  if (gx > 8192) gx = 8192;
  if (gx < 1) gx = 1;
  return dim3((unsigned)gx, (unsigned)((chunks + cpb - 1) / cpb));
}

// ---------------------------------------------------------------- column reductions
// the finished column sums of one column, by mode
XP_DEV void col_finish_one(const ColArgs& a, int col, double s0, double s1) {
  if (a.mode == COL_STATS) {
    bn_stats_from_sums(s0, s1, a.M, a.eps, a.out0 + col, a.out1 + col);
  } else if (a.mode == COL_BNBWD) {
    a.out0[col] = s0;
    a.out1[col] = s1;
    a.grad0[col] = (float)((double)a.grad0[col] + s1);
    a.grad1[col] = (float)((double)a.grad1[col] + s0);
  } else {
    a.grad0[col] = (float)((double)a.grad0[col] + s0);
  }
}

// Block: CL chunk-lanes x RG row groups; partials per (row block, column);
// the row groups of a block are added in a fixed order in LDS.
template <typename T>
__global__ __launch_bounds__(256) void k_colpart_v(ColArgs a) {
  constexpr int N = VT<T>::N;
  __shared__ double sh[2][256][N];
  const int chunks = a.C / N;
  const int CL = chunks < 256 ? chunks : 256;
  const int RG = 256 / CL;
  const int cl = threadIdx.x % CL, g = threadIdx.x / CL;
  const int chunk = blockIdx.x * CL + cl;
  const int per = ceil_div(a.M, a.row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(a.M, r0 + per);
  const T* A = (const T*)a.a;
  const T* Z = (const T*)a.z;
  double s0[N], s1[N];
#pragma unroll
  for (int e = 0; e < N; ++e) s0[e] = s1[e] = 0.0;
  if (g < RG && chunk < chunks) {
    const int c0 = chunk * N;
    double mu[N], rs[N];
    if (a.mode == COL_BNBWD) {
#pragma unroll
      for (int e = 0; e < N; ++e) { mu[e] = a.mean[c0 + e]; rs[e] = a.rstd[c0 + e]; }
    }
    // rows r0 + g, r0 + g + RG, ... in order, four per trip with the trip's
    // loads issued first
    constexpr int U = 4;
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    for (int rb = r0 + g; rb < r1; rb += U * RG) {
      uint4 av[U], zv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = rb + u * RG;
        av[u] = zv[u] = zero;
        if (r < r1) {
          av[u] = ld16(A + (size_t)r * a.lda + c0);
          if (a.mode == COL_BNBWD) zv[u] = ld16(Z + (size_t)r * a.ldz + c0);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (rb + u * RG >= r1) break;
        double v[N];
        cvt16<T>(av[u], v);
        if (a.mode == COL_STATS) {
#pragma unroll
          for (int e = 0; e < N; ++e) { s0[e] += v[e]; s1[e] += v[e] * v[e]; }
        } else if (a.mode == COL_BNBWD) {
          double z[N];
          cvt16<T>(zv[u], z);
#pragma unroll
          for (int e = 0; e < N; ++e) { s0[e] += v[e]; s1[e] += v[e] * ((z[e] - mu[e]) * rs[e]); }
        } else {
#pragma unroll
          for (int e = 0; e < N; ++e) s0[e] += v[e];
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < N; ++e) { sh[0][threadIdx.x][e] = s0[e]; sh[1][threadIdx.x][e] = s1[e]; }
  // the RG row groups of a column are added pairwise in a fixed tree: at each
  // level group g takes in group g + half
  int half = 1;
  while (2 * half < RG) half *= 2;
  for (; half >= 1; half >>= 1) {
    __syncthreads();
    if (g < half && g + half < RG) {
      const int o = (g + half) * CL + cl;
#pragma unroll
      for (int e = 0; e < N; ++e) {
        sh[0][threadIdx.x][e] += sh[0][o][e];
        sh[1][threadIdx.x][e] += sh[1][o][e];
      }
    }
  }
  if (g == 0 && chunk < chunks) {
    const int c0 = chunk * N;
#pragma unroll
    for (int e = 0; e < N; ++e) {
      a.partial[((size_t)(c0 + e) * 2 + 0) * a.row_blocks + blockIdx.y] = sh[0][cl][e];
      a.partial[((size_t)(c0 + e) * 2 + 1) * a.row_blocks + blockIdx.y] = sh[1][cl][e];
    }
  }
}

// finalize: one workgroup per column; the partials of a column are contiguous,
// each thread adds a fixed stride of them, then the waves and the block add in
// a fixed order
__global__ __launch_bounds__(256) void k_colfinal_v(ColArgs a) {
  __shared__ double sh[2][4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.x;
  const double* p0 = a.partial + (size_t)col * 2 * a.row_blocks;
  const double* p1 = p0 + a.row_blocks;
  // the gradient accumulators the finish adds to, read before the reduction
  // so that their latency overlaps it
  float acc0 = 0.f, acc1 = 0.f;
  if (threadIdx.x == 0 && a.mode != COL_STATS) {
    acc0 = a.grad0[col];
    if (a.mode == COL_BNBWD) acc1 = a.grad1[col];
  }
  double s0 = 0.0, s1 = 0.0;
#pragma unroll 4
  for (int b = threadIdx.x; b < a.row_blocks; b += 256) {
    s0 += p0[b];
    s1 += p1[b];
  }
  s0 = wave_sum(s0);
  s1 = wave_sum(s1);
  if (lane == 0) {
    sh[0][wave] = s0;
    sh[1][wave] = s1;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double t0 = ((sh[0][0] + sh[0][1]) + sh[0][2]) + sh[0][3];
    const double t1 = ((sh[1][0] + sh[1][1]) + sh[1][2]) + sh[1][3];
    if (a.mode == COL_STATS) {
      col_finish_one(a, col, t0, t1);
    } else if (a.mode == COL_BNBWD) {
      a.out0[col] = t0;
      a.out1[col] = t1;
      a.grad0[col] = (float)((double)acc0 + t1);
      a.grad1[col] = (float)((double)acc1 + t0);
    } else {
      a.grad0[col] = (float)((double)acc0 + t0);
    }
  }
}

hipError_t launch_colfinal(const ColArgs& a, hipStream_t s) {
  if (a.C <= 0) return hipSuccess;
  XP_LAUNCH("k_colfinal_v", (double)a.row_blocks * 2 * a.C * 8, k_colfinal_v, dim3(a.C),
            dim3(256), 0, s, a);
  return hipGetLastError();
}

int col_row_blocks_v(int M, int C, int N) {
  int chunks = C / N;
  int CL = chunks < 256 ? chunks : 256;
  int RG = 256 / CL;
  int colblocks = ceil_div(chunks, CL);
  int want = ceil_div(1024, colblocks);         // ~1024 workgroups: every CU busy
  int maxrb = ceil_div(M, RG * 4);              // >= ~4 rows per thread
  if (want > maxrb) want = maxrb;
  if (want > COL_MAX_ROW_BLOCKS_V) want = COL_MAX_ROW_BLOCKS_V;
  return want < 1 ? 1 : want;
}

template <typename T>
static hipError_t colreduce_v(ColArgs a, hipStream_t s) {
  constexpr int N = VT<T>::N;
  int chunks = a.C / N;
  int CL = chunks < 256 ? chunks : 256;
  a.row_blocks = col_row_blocks_v(a.M, a.C, N);
  XP_LAUNCH(sizeof(T) == 2 ? "k_colpart_v<bf16>" : "k_colpart_v<f32>",
            (double)a.M * a.C * sizeof(T) * (a.mode == COL_BNBWD ? 2 : 1), k_colpart_v<T>,
            dim3(ceil_div(chunks, CL), a.row_blocks), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_colfinal(a, s);
}


// ---------------------------------------------------------------- BN apply / backward
template <typename T, int U>
__global__ __launch_bounds__(256) void k_bn_apply_v(BnApplyArgs a) {
  constexpr int N = VT<T>::N;
  const RowMap m = row_map<T>(a.C);
  if (!m.live) return;
  const int c0 = m.chunk * N;
  // one BN, or the BN whose channel range holds this chunk (y, gamma and beta
  // then start at the range's first channel)
  T* Y = (T*)a.y;
  int ldy = a.ldy, yc = c0, relu = a.relu;
  const float* gam = a.gamma + c0;
  const float* bet = a.beta + c0;
  if (a.nseg > 0) {
    bool found = false;
#pragma unroll
    for (int q = 0; q < BN_APPLY_SEGS; ++q)
      if (q < a.nseg && c0 >= a.seg_c0[q] && c0 < a.seg_c1[q]) {
        found = true;
        Y = (T*)a.seg_y[q];
        ldy = a.seg_ldy[q];
        yc = c0 - a.seg_c0[q];
        relu = a.seg_relu[q];
        gam = a.seg_gamma[q] + yc;
        bet = a.seg_beta[q] + yc;
      }
    if (!found) return;
  }
  double mu[N], rs[N], ga[N], be[N];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    mu[e] = a.mean[c0 + e];
    rs[e] = a.rstd[c0 + e];
    ga[e] = (double)gam[e];
    be[e] = (double)bet[e];
  }
  const T* Z = (const T*)a.z;
  const T* R = (const T*)a.res;
  for (int r0 = m.row0; r0 < a.M; r0 += U * m.stride) {
    uint4 zr[U], rr[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * m.stride;
      zr[u] = rr[u] = make_uint4(0u, 0u, 0u, 0u);
      if (r < a.M) {
        zr[u] = ld16(Z + (size_t)r * a.ldz + c0);
        if (R) rr[u] = ld16(R + (size_t)r * a.ldres + c0);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * m.stride;
      if (r >= a.M) break;
      double z[N], q[N];
      cvt16<T>(zr[u], z);
      if (R) cvt16<T>(rr[u], q);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        double xh = (z[e] - mu[e]) * rs[e];
        double v = ga[e] * xh + be[e];
        // the BN output is rounded to the storage type before the residual add
        if (R) v = rnd<T>(v) + q[e];
        if (relu) v = v > 0.0 ? v : 0.0;
        z[e] = v;
      }
      vst(Y + (size_t)r * ldy + yc, z);
    }
  }
}

template <typename T, int U>
__global__ __launch_bounds__(256) void k_bn_bwd_v(BnBwdArgs a) {
  constexpr int N = VT<T>::N;
  const RowMap m = row_map<T>(a.C);
  if (!m.live) return;
  const int c0 = m.chunk * N;
  // d = gamma rstd (g - dbeta / M - xh dgamma / M), xh = (z - mean) rstd
  double mu[N], rs[N], grs[N], db[N], dg[N];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const int c = c0 + e;
    mu[e] = a.mean[c];
    rs[e] = a.rstd[c];
    grs[e] = (double)a.gamma[c] * rs[e];
    db[e] = a.dbeta[c] / a.M;
    dg[e] = a.dgamma[c] / a.M;
  }
  const T* G = (const T*)a.g;
  const T* Z = (const T*)a.z;
  T* DZ = (T*)a.dz;
  T* DR = (T*)a.dres;
  const T* RM = (const T*)a.resmask;
  const T* ZM = (const T*)a.dzmask;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  // the residual source can be the BN input itself (its gradient accumulates
  // onto the BN-input gradient just stored): then the stored chunk is reused
  const bool res_is_dz = DR == DZ && a.lddres == a.lddz;
  for (int r0 = m.row0; r0 < a.M; r0 += U * m.stride) {
    uint4 gr[U], zr[U], zm[U], zo[U], rm[U], ro[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * m.stride;
      gr[u] = zr[u] = zm[u] = zo[u] = rm[u] = ro[u] = zero;
      if (r < a.M) {
        gr[u] = ld16(G + (size_t)r * a.ldg + c0);
        zr[u] = ld16(Z + (size_t)r * a.ldz + c0);
        if (ZM) zm[u] = ld16(ZM + (size_t)r * a.ldzm + c0);
        if (a.dz_accumulate) zo[u] = ld16(DZ + (size_t)r * a.lddz + c0);
        if (DR && RM) rm[u] = ld16(RM + (size_t)r * a.ldrm + c0);
        if (DR && a.res_accumulate && !res_is_dz) ro[u] = ld16(DR + (size_t)r * a.lddres + c0);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * m.stride;
      if (r >= a.M) break;
      double g[N], z[N], d[N];
      cvt16<T>(gr[u], g);
      cvt16<T>(zr[u], z);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        double xh = (z[e] - mu[e]) * rs[e];
        d[e] = grs[e] * (g[e] - db[e] - xh * dg[e]);
      }
      if (ZM) vmask_raw<T>(zm[u], d);
      if (a.dz_accumulate) {
        double o[N];
        cvt16<T>(zo[u], o);
#pragma unroll
        for (int e = 0; e < N; ++e) d[e] += o[e];
      }
      const uint4 dbits = pack16<T>(d);
      *reinterpret_cast<uint4*>(DZ + (size_t)r * a.lddz + c0) = dbits;
      if (DR) {
        if (RM) vmask_raw<T>(rm[u], g);
        if (a.res_accumulate) {
          double o[N];
          cvt16<T>(res_is_dz ? dbits : ro[u], o);
#pragma unroll
          for (int e = 0; e < N; ++e) g[e] += o[e];
        }
        vst(DR + (size_t)r * a.lddres + c0, g);
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_elt_v(EltArgs a) {
  constexpr int N = VT<T>::N;
  const int chunks = a.C / N;
  const int items = a.M * chunks;
  const T* A = (const T*)a.a;
  const T* B = (const T*)a.b;
  const T* MK = (const T*)a.mask;
  T* Y = (T*)a.y;
  for (int it = blockIdx.x * blockDim.x + threadIdx.x; it < items; it += gridDim.x * blockDim.x) {
    const int r = it / chunks, c0 = (it - r * chunks) * N;
    double v[N];
    vld(A + (size_t)r * a.lda + c0, v);
    if (B) {
      double b[N];
      vld(B + (size_t)r * a.ldb + c0, b);
#pragma unroll
      for (int e = 0; e < N; ++e) v[e] += b[e];
    }
    if (a.relu) {
#pragma unroll
      for (int e = 0; e < N; ++e) v[e] = v[e] > 0.0 ? v[e] : 0.0;
    }
    if (MK) vmask(MK + (size_t)r * a.ldm + c0, v);
    T* p = Y + (size_t)r * a.ldy + c0;
    if (a.accumulate) {
      double o[N];
      vld(p, o);
#pragma unroll
      for (int e = 0; e < N; ++e) v[e] += o[e];
    }
    vst(p, v);
  }
}

// ---------------------------------------------------------------- pooling
template <typename T>
__global__ __launch_bounds__(256) void k_maxpool_fwd_v(PoolArgs a) {
  constexpr int N = VT<T>::N;
  const int chunks = a.C / N, Ho = a.H / 2, Wo = a.W / 2;
  const int items = a.nb * Ho * Wo * chunks;
  const T* X = (const T*)a.x;
  T* O = (T*)a.out;
  for (int it = blockIdx.x * blockDim.x + threadIdx.x; it < items; it += gridDim.x * blockDim.x) {
    const int r = it / chunks, c0 = (it - r * chunks) * N;
    const int n = r / (Ho * Wo), rem = r - n * Ho * Wo, ho = rem / Wo, wo = rem - ho * Wo;
    const T* base = X + ((size_t)(n * a.H + 2 * ho) * a.W + 2 * wo) * a.ldx + c0;
    double b[N], q[N];
    vld(base, b);
    const T* others[3] = {base + a.ldx, base + (size_t)a.W * a.ldx, base + ((size_t)a.W + 1) * a.ldx};
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      vld(others[k], q);
#pragma unroll
      for (int e = 0; e < N; ++e)
        if (q[e] > b[e]) b[e] = q[e];
    }
    vst(O + (size_t)r * a.ldo + c0, b);  // a max of stored values is stored exactly
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_maxpool_bwd_v(PoolArgs a) {
  constexpr int N = VT<T>::N;
  const int chunks = a.C / N, Ho = a.H / 2, Wo = a.W / 2;
  const int items = a.nb * a.H * a.W * chunks;
  const T* X = (const T*)a.x;
  const T* DY = (const T*)a.dy;
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  for (int it = blockIdx.x * blockDim.x + threadIdx.x; it < items; it += gridDim.x * blockDim.x) {
    const int r = it / chunks, c0 = (it - r * chunks) * N;
    const int n = r / (a.H * a.W), rem = r - n * a.H * a.W, h = rem / a.W, w = rem - h * a.W;
    const int ho = h >> 1, wo = w >> 1;
    double d[N];
#pragma unroll
    for (int e = 0; e < N; ++e) d[e] = 0.0;
    if (ho < Ho && wo < Wo) {
      const T* base = X + ((size_t)(n * a.H + 2 * ho) * a.W + 2 * wo) * a.ldx + c0;
      double v[4][N];
      vld(base, v[0]);
      vld(base + a.ldx, v[1]);
      vld(base + (size_t)a.W * a.ldx, v[2]);
      vld(base + ((size_t)a.W + 1) * a.ldx, v[3]);
      double g[N];
      vld(DY + ((size_t)(n * Ho + ho) * Wo + wo) * a.lddy + c0, g);
      const int me = ((h & 1) << 1) + (w & 1);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        // the running maximum is kept by value (no runtime index into v)
        int arg = 0;
        double best = v[0][e];
#pragma unroll
        for (int q = 1; q < 4; ++q)
          if (v[q][e] > best) {  // first maximum in row-major order wins ties
            best = v[q][e];
            arg = q;
          }
        d[e] = arg == me ? g[e] : 0.0;
      }
    }
    if (MK) vmask(MK + (size_t)r * a.ldm + c0, d);
    T* p = O + (size_t)r * a.ldo + c0;
    if (a.accumulate) {
      double o[N];
      vld(p, o);
#pragma unroll
      for (int e = 0; e < N; ++e) d[e] += o[e];
    }
    vst(p, d);
  }
}

// 3x3 / stride 1 / zero-padded average (padding counted): each thread owns a
// run of AVG_SEG outputs of one image row and one 16-byte channel chunk.  It
// issues every load of its 3 x (AVG_SEG + 2) input window (and of its mask and
// accumulation operands) before any arithmetic, so a thread waits on memory
// once, then slides along the run keeping the vertical three-row sums of the
// previous, current and next column:
// out(h, w) = ((v(w-1) + v(w)) + v(w+1)) / 9, v(w) = (x(h-1, w) + x(h, w)) + x(h+1, w),
// with zeros outside the image.  The kernel is bound by its arithmetic, not by
// memory: fp32 storage computes in fp64 (one rounding on store, as everywhere
// in that variant); bf16 storage computes in fp32, like the bf16 variant's
// accumulations, at twice the rate and without conversions to fp64, and takes
// the ninth as a product with the fp32 reciprocal of 9 (within an fp32 ulp of
// the quotient, far below the bf16 rounding it is followed by; the quotient's
// division sequence was most of the kernel's arithmetic).
template <typename T> struct AvgAcc {
  typedef double t;
  static XP_DEV double ninth(double v) { return v / 9.0; }
};
template <> struct AvgAcc<bf16_t> {
  typedef float t;
  static XP_DEV float ninth(float v) { return v * (1.0f / 9.0f); }
};
// runs of 4 outputs: 3 x 6 window chunks in registers keep three waves per
// SIMD resident (runs of 7 needed 181 VGPRs, two waves): 13.8 -> 12.4 us per
// launch on the Inception-A stage (runs of 5: 12.9); the blocks go to the
// XCDs in contiguous runs (13.8 -> 14.6 us without)
constexpr int AVG_SEG = 4;
template <typename T>
__global__ __launch_bounds__(256) void k_avgpool3_v(PoolArgs a, const T* src, int ld_src) {
  constexpr int N = VT<T>::N;
  constexpr int WIN = AVG_SEG + 2;
  const int chunks = a.C / N;
  const int nseg = ceil_div(a.W, AVG_SEG);
  // XCD-contiguous block order: the three output rows that read an input row
  // run in one XCD's L2
  int it = xcd_tile(blockIdx.x, gridDim.x) * blockDim.x + threadIdx.x;
  if (it >= a.nb * a.H * nseg * chunks) return;
  const int chunk = it % chunks;
  it /= chunks;
  const int seg = it % nseg;
  it /= nseg;
  const int h = it % a.H, n = it / a.H;
  const int c0 = chunk * N;
  const int w0 = seg * AVG_SEG;
  const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
  uint4 win[3][WIN];
#pragma unroll
  for (int dr = 0; dr < 3; ++dr) {
    const int hh = h + dr - 1;
    const bool rok = hh >= 0 && hh < a.H;
#pragma unroll
    for (int j = 0; j < WIN; ++j) {
      const int w = w0 - 1 + j;
      win[dr][j] = (rok && w >= 0 && w < a.W)
                       ? ld16(src + ((size_t)(n * a.H + hh) * a.W + w) * ld_src + c0) : zero;
    }
  }
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  const size_t rbase = (size_t)(n * a.H + h) * a.W;
  uint4 mk[AVG_SEG], old[AVG_SEG];
#pragma unroll
  for (int j = 0; j < AVG_SEG; ++j) {
    mk[j] = old[j] = zero;
    if (w0 + j < a.W) {
      if (MK) mk[j] = ld16(MK + (rbase + w0 + j) * a.ldm + c0);
      if (a.accumulate) old[j] = ld16(O + (rbase + w0 + j) * a.ldo + c0);
    }
  }
  typedef typename AvgAcc<T>::t A;
  auto cvt = [&](uint4 u, A* v) {
    if constexpr (sizeof(T) == 2) {
      const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(wd[i] << 16);
        v[2 * i + 1] = __uint_as_float(wd[i] & 0xffff0000u);
      }
    } else {
      cvt16<T>(u, v);
    }
  };
  auto vsum = [&](int j, A* v) {
    A q0[N], q1[N], q2[N];
    cvt(win[0][j], q0);
    cvt(win[1][j], q1);
    cvt(win[2][j], q2);
#pragma unroll
    for (int e = 0; e < N; ++e) v[e] = (q0[e] + q1[e]) + q2[e];
  };
  A vp[N], vc[N], vn[N];
  vsum(0, vp);
  vsum(1, vc);
#pragma unroll
  for (int j = 0; j < AVG_SEG; ++j) {
    if (w0 + j >= a.W) break;
    vsum(j + 2, vn);
    double s[N];
#pragma unroll
    for (int e = 0; e < N; ++e) s[e] = (double)AvgAcc<T>::ninth((vp[e] + vc[e]) + vn[e]);
    if (MK) vmask_raw<T>(mk[j], s);
    if (a.accumulate) {
      double q[N];
      cvt16<T>(old[j], q);
#pragma unroll
      for (int e = 0; e < N; ++e) s[e] += q[e];
    }
    vst(O + (rbase + w0 + j) * a.ldo + c0, s);
#pragma unroll
    for (int e = 0; e < N; ++e) {
      vp[e] = vc[e];
      vc[e] = vn[e];
    }
  }
}

// 3x3 / stride 2 max pool, padding p = 1 (never chosen: the window centre
// (2ho, 2wo) is always inside) or 0 (valid), over groups of N channels
// (16-byte chunks, or single channels).  Ties go to the first maximum in
// row-major window order (strict > while scanning).
template <typename T, int N>
XP_DEV void ldn(const T* p, double* v) {
  if constexpr (N == VT<T>::N) vld(p, v);
  else
#pragma unroll
    for (int e = 0; e < N; ++e) v[e] = ldd(p + e);
}
template <typename T, int N>
XP_DEV void stn(T* p, const double* v) {
  if constexpr (N == VT<T>::N) vst(p, v);
  else
#pragma unroll
    for (int e = 0; e < N; ++e) std_(p + e, v[e]);
}

template <typename T, int N>
__global__ __launch_bounds__(256) void k_maxpool3s2_fwd(PoolArgs a, int Ho, int Wo) {
  const int groups = a.C / N;
  int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (it >= (int64_t)a.nb * Ho * Wo * groups) return;
  const int g = (int)(it % groups);
  it /= groups;
  const int wo = (int)(it % Wo);
  it /= Wo;
  const int ho = (int)(it % Ho), n = (int)(it / Ho);
  const int c0 = g * N;
  const T* X = (const T*)a.x;
  const int p = a.valid ? 0 : 1;
  double best[N];
  uint32_t pos[N];  // window position of the first maximum
  bool have = false;
  for (int r = 0; r < 3; ++r) {
    const int h = 2 * ho - p + r;
    if (h < 0 || h >= a.H) continue;
    for (int q = 0; q < 3; ++q) {
      const int w = 2 * wo - p + q;
      if (w < 0 || w >= a.W) continue;
      double v[N];
      ldn<T, N>(X + ((size_t)(n * a.H + h) * a.W + w) * a.ldx + c0, v);
#pragma unroll
      for (int e = 0; e < N; ++e)
        if (!have || v[e] > best[e]) {
          best[e] = v[e];
          pos[e] = (uint32_t)(r * 3 + q);
        }
      have = true;
    }
  }
  const size_t o = (size_t)(n * Ho + ho) * Wo + wo;
  stn<T, N>((T*)a.out + o * a.ldo + c0, best);
  if (a.idx) {
    // a NaN maximum chooses no position (0xff matches none)
#pragma unroll
    for (int e = 0; e < N; ++e)
      if (best[e] != best[e]) pos[e] = 0xffu;
    uint8_t* ip = a.idx + o * a.ldi + c0;
    if constexpr (N == 8) {
      uint2 v;
      v.x = pos[0] | (pos[1] << 8) | (pos[2] << 16) | (pos[3] << 24);
      v.y = pos[4] | (pos[5] << 8) | (pos[6] << 16) | (pos[7] << 24);
      *reinterpret_cast<uint2*>(ip) = v;
    } else if constexpr (N == 4) {
      *reinterpret_cast<uint32_t*>(ip) = pos[0] | (pos[1] << 8) | (pos[2] << 16) | (pos[3] << 24);
    } else {
#pragma unroll
      for (int e = 0; e < N; ++e) ip[e] = (uint8_t)pos[e];
    }
  }
}

// backward: each input pixel gathers, in (ho, wo) order, the output gradients
// of the (at most four) windows that contain it and chose it: the forward
// recorded, per window and channel, the position of its first maximum.
template <typename T, int N>
__global__ __launch_bounds__(256) void k_maxpool3s2_bwd(PoolArgs a, int Ho, int Wo) {
  const int groups = a.C / N;
  int64_t it = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (it >= (int64_t)a.nb * a.H * a.W * groups) return;
  const int g = (int)(it % groups);
  it /= groups;
  const int w = (int)(it % a.W);
  it /= a.W;
  const int h = (int)(it % a.H), n = (int)(it / a.H);
  const int c0 = g * N;
  const T* DY = (const T*)a.dy;
  const int pd = a.valid ? 0 : 1;
  double acc[N];
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.0;
  // windows 2ho - pd .. 2ho - pd + 2 that contain row h: ho from ceil((h + pd - 2) / 2)
  const int ho0 = max(0, (h + pd - 1) / 2), wo0 = max(0, (w + pd - 1) / 2);
  const int ho1 = min((h + pd) / 2, Ho - 1), wo1 = min((w + pd) / 2, Wo - 1);
  // the forward's choice: this pixel's position in each covering window
  for (int ho = ho0; ho <= ho1; ++ho)
    for (int wo = wo0; wo <= wo1; ++wo) {
      const size_t o = (size_t)(n * Ho + ho) * Wo + wo;
      const uint32_t me = (uint32_t)((h - (2 * ho - pd)) * 3 + (w - (2 * wo - pd)));
      const uint8_t* ip = a.idx + o * a.ldi + c0;
      uint32_t pos[N];
      if constexpr (N == 8) {
        const uint2 v = *reinterpret_cast<const uint2*>(ip);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pos[e] = (v.x >> (8 * e)) & 0xffu;
          pos[e + 4] = (v.y >> (8 * e)) & 0xffu;
        }
      } else if constexpr (N == 4) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(ip);
#pragma unroll
        for (int e = 0; e < 4; ++e) pos[e] = (v >> (8 * e)) & 0xffu;
      } else {
#pragma unroll
        for (int e = 0; e < N; ++e) pos[e] = ip[e];
      }
      double d[N];
      ldn<T, N>(DY + o * a.lddy + c0, d);
#pragma unroll
      for (int e = 0; e < N; ++e)
        if (pos[e] == me) acc[e] += d[e];
    }
  const size_t r = (size_t)(n * a.H + h) * a.W + w;
  if (a.mask) {
    double m[N];
    ldn<T, N>((const T*)a.mask + r * a.ldm + c0, m);
#pragma unroll
    for (int e = 0; e < N; ++e)
      if (!(m[e] > 0.0)) acc[e] = 0.0;
  }
  T* p = (T*)a.out + r * a.ldo + c0;
  if (a.accumulate) {
    double o[N];
    ldn<T, N>(p, o);
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] += o[e];
  }
  stn<T, N>(p, acc);
}

template <typename T>
static hipError_t maxpool3s2_go(const PoolArgs& a, bool bwd, hipStream_t s) {
  const int p = a.valid ? 0 : 1;
  const int Ho = (a.H + 2 * p - 3) / 2 + 1, Wo = (a.W + 2 * p - 3) / 2 + 1;
  if (Ho <= 0 || Wo <= 0) return hipErrorInvalidValue;
  constexpr int V = VT<T>::N;
  const bool vec = vec_ok<T>(a.C, {{a.x, a.ldx}, {a.out, a.ldo}, {a.dy, a.lddy}, {a.mask, a.ldm},
                                   {a.y, a.ldy}});
  // the backward reads the positions the forward recorded
  if (bwd && !a.idx) return hipErrorInvalidValue;
  // indices are stored as one byte per channel, N-byte groups aligned
  if (a.idx && (a.ldi < a.C || (vec && ((a.ldi % VT<T>::N) != 0 ||
                                       (reinterpret_cast<uintptr_t>(a.idx) % VT<T>::N) != 0))))
    return hipErrorInvalidValue;
  const int64_t pix = bwd ? (int64_t)a.nb * a.H * a.W : (int64_t)a.nb * Ho * Wo;
  const int64_t threads = pix * (vec ? a.C / V : a.C);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  const double esz = sizeof(T);
  // algorithmic bytes: forward reads x once and writes y; backward reads x, dy
  // (and mask / old dx) and writes dx
  const double in_b = (double)a.nb * a.H * a.W * a.C * esz, out_b = (double)a.nb * Ho * Wo * a.C * esz;
  const double bytes = bwd ? 2 * in_b + out_b + (a.mask ? in_b : 0) + (a.accumulate ? in_b : 0)
                           : in_b + out_b;
  const char* name = bwd ? (sizeof(T) == 2 ? "k_maxpool3s2_bwd<bf16>" : "k_maxpool3s2_bwd<f32>")
                         : (sizeof(T) == 2 ? "k_maxpool3s2_fwd<bf16>" : "k_maxpool3s2_fwd<f32>");
  if (vec) {
    if (bwd) XP_LAUNCH(name, bytes, (k_maxpool3s2_bwd<T, V>), dim3(blocks), dim3(256), 0, s, a, Ho, Wo);
    else XP_LAUNCH(name, bytes, (k_maxpool3s2_fwd<T, V>), dim3(blocks), dim3(256), 0, s, a, Ho, Wo);
  } else {
    if (bwd) XP_LAUNCH(name, bytes, (k_maxpool3s2_bwd<T, 1>), dim3(blocks), dim3(256), 0, s, a, Ho, Wo);
    else XP_LAUNCH(name, bytes, (k_maxpool3s2_fwd<T, 1>), dim3(blocks), dim3(256), 0, s, a, Ho, Wo);
  }
  return hipGetLastError();
}

hipError_t launch_maxpool3s2_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  if (a.nb <= 0 || a.H <= 0 || a.W <= 0 || a.C <= 0) return hipSuccess;
  return dtype == DT_BF16 ? maxpool3s2_go<bf16_t>(a, false, s) : maxpool3s2_go<float>(a, false, s);
}
hipError_t launch_maxpool3s2_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  if (a.nb <= 0 || a.H <= 0 || a.W <= 0 || a.C <= 0) return hipSuccess;
  return dtype == DT_BF16 ? maxpool3s2_go<bf16_t>(a, true, s) : maxpool3s2_go<float>(a, true, s);
}

// Global average pool, two launches: per (image, pixel split) partial sums of
// every channel (fixed order: strided per thread, then the row groups in
// order), then per (image, channel) the splits in order, divided by H*W.
template <typename T>
__global__ __launch_bounds__(256) void k_gap_part_v(PoolArgs a, int splits) {
  constexpr int N = VT<T>::N;
  __shared__ double sh[256][N];
  const int chunks = a.C / N;
  const int CL = chunks < 256 ? chunks : 256;
  const int RG = 256 / CL;
  const int cl = threadIdx.x % CL, g = threadIdx.x / CL;
  const int chunk = blockIdx.z * CL + cl;
  const int split = blockIdx.x, n = blockIdx.y;
  const int HW = a.H * a.W;
  const int per = ceil_div(HW, splits);
  const int p0 = split * per, p1 = min(HW, p0 + per);
  const T* X = (const T*)a.x;
  double s[N];
#pragma unroll
  for (int e = 0; e < N; ++e) s[e] = 0.0;
  if (g < RG && chunk < chunks) {
#pragma unroll 4
    for (int p = p0 + g; p < p1; p += RG) {
      double q[N];
      vld(X + ((size_t)n * HW + p) * a.ldx + chunk * N, q);
#pragma unroll
      for (int e = 0; e < N; ++e) s[e] += q[e];
    }
  }
#pragma unroll
  for (int e = 0; e < N; ++e) sh[threadIdx.x][e] = s[e];
  __syncthreads();
  if (g == 0 && chunk < chunks) {
    double t[N];
#pragma unroll
    for (int e = 0; e < N; ++e) t[e] = 0.0;
    for (int q = 0; q < RG; ++q)
#pragma unroll
      for (int e = 0; e < N; ++e) t[e] += sh[q * CL + cl][e];
    double* P = a.part + ((size_t)n * splits + split) * a.C + chunk * N;
#pragma unroll
    for (int e = 0; e < N; ++e) P[e] = t[e];
  }
}

// one wave per (image, channel chunk): lane q holds split q, the wave adds the
// splits in a fixed butterfly order
template <typename T>
__global__ __launch_bounds__(256) void k_gap_fin_v(PoolArgs a, int splits) {
  constexpr int N = VT<T>::N;
  const int chunks = a.C / N;
  const int lane = threadIdx.x & 63;
  const int it = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (it >= a.nb * chunks) return;
  const int n = it / chunks, c0 = (it - n * chunks) * N;
  double t[N];
#pragma unroll
  for (int e = 0; e < N; ++e) t[e] = 0.0;
  if (lane < splits) {
    const double* P = a.part + ((size_t)n * splits + lane) * a.C + c0;
#pragma unroll
    for (int e = 0; e < N; ++e) t[e] = P[e];
  }
#pragma unroll
  for (int e = 0; e < N; ++e) t[e] = wave_sum(t[e]) / (a.H * a.W);
  if (lane == 0) vst((T*)a.out + (size_t)n * a.ldo + c0, t);
}

template <typename T>
__global__ __launch_bounds__(256) void k_gap_bwd_v(PoolArgs a) {
  constexpr int N = VT<T>::N;
  const int chunks = a.C / N;
  const int HW = a.H * a.W;
  const int items = a.nb * HW * chunks;
  const T* DY = (const T*)a.dy;
  const T* MK = (const T*)a.mask;
  T* O = (T*)a.out;
  for (int it = blockIdx.x * blockDim.x + threadIdx.x; it < items; it += gridDim.x * blockDim.x) {
    const int r = it / chunks, c0 = (it - r * chunks) * N;
    const int n = r / HW;
    double d[N];
    vld(DY + (size_t)n * a.lddy + c0, d);
#pragma unroll
    for (int e = 0; e < N; ++e) d[e] = d[e] / HW;
    if (MK) vmask(MK + (size_t)r * a.ldm + c0, d);
    T* p = O + (size_t)r * a.ldo + c0;
    if (a.accumulate) {
      double o[N];
      vld(p, o);
#pragma unroll
      for (int e = 0; e < N; ++e) d[e] += o[e];
    }
    vst(p, d);
  }
}

// GAP backward with batch-norm backward partials: blocks of CL chunk-lanes x
// RG row groups over a row block, as the column partials are laid out; each
// thread forms g = dy / (H W) for its chunk's rows (masked, added to the
// stored value when accumulating), stores it, and adds the stored values and
// their products with (z - mean) rstd; the row groups are then added in a
// fixed pairwise tree
template <typename T>
__global__ __launch_bounds__(256) void k_gap_bwd_bn_v(PoolArgs a, GapBnArgs b, int row_blocks) {
  constexpr int N = VT<T>::N;
  __shared__ double sh[2][256][N];
  const int chunks = a.C / N;
  const int CL = chunks < 256 ? chunks : 256;
  const int RG = 256 / CL;
  const int cl = threadIdx.x % CL, g = threadIdx.x / CL;
  const int chunk = blockIdx.x * CL + cl;
  const int HW = a.H * a.W, M = a.nb * HW;
  const int per = ceil_div(M, row_blocks);
  const int r0 = blockIdx.y * per, r1 = min(M, r0 + per);
  double s0[N], s1[N];
#pragma unroll
  for (int e = 0; e < N; ++e) s0[e] = s1[e] = 0.0;
  if (g < RG && chunk < chunks) {
    const int c0 = chunk * N;
    // this chunk's norm (selected with constant indices)
    const T* Z = nullptr;
    int ldz = 0;
    const double *mp = nullptr, *rp = nullptr;
#pragma unroll
    for (int q = 0; q < CONV_BN_SEGS; ++q)
      if (q < b.bn_nseg && c0 >= b.bn_c0[q] && c0 < b.bn_c1[q]) {
        const int lc = c0 - b.bn_c0[q];
        Z = (const T*)b.bn_z[q] + lc;
        ldz = b.ld_bnz[q];
        mp = b.bn_mean[q] + lc;
        rp = b.bn_rstd[q] + lc;
      }
    double mu[N], rs[N];
#pragma unroll
    for (int e = 0; e < N; ++e) {
      mu[e] = Z ? mp[e] : 0.0;
      rs[e] = Z ? rp[e] : 0.0;
    }
    const T* DY = (const T*)a.dy;
    const T* MK = (const T*)a.mask;
    T* O = (T*)a.out;
    constexpr int U = 4;
    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
    for (int rb = r0 + g; rb < r1; rb += U * RG) {
      uint4 dv[U], mv[U], ov[U], zv[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = rb + u * RG;
        dv[u] = mv[u] = ov[u] = zv[u] = zero;
        if (r < r1) {
          dv[u] = ld16(DY + (size_t)(r / HW) * a.lddy + c0);
          if (MK) mv[u] = ld16(MK + (size_t)r * a.ldm + c0);
          if (a.accumulate) ov[u] = ld16(O + (size_t)r * a.ldo + c0);
          if (Z) zv[u] = ld16(Z + (size_t)r * ldz);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = rb + u * RG;
        if (r >= r1) break;
        double d[N];
        cvt16<T>(dv[u], d);
#pragma unroll
        for (int e = 0; e < N; ++e) d[e] = d[e] / HW;
        if (MK) vmask_raw<T>(mv[u], d);
        if (a.accumulate) {
          double o[N];
          cvt16<T>(ov[u], o);
#pragma unroll
          for (int e = 0; e < N; ++e) d[e] += o[e];
        }
        const uint4 st = pack16<T>(d);
        *reinterpret_cast<uint4*>(O + (size_t)r * a.ldo + c0) = st;
        if (Z) {
          double v[N], z[N];
          cvt16<T>(st, v);  // the stored values
          cvt16<T>(zv[u], z);
#pragma unroll
          for (int e = 0; e < N; ++e) {
            s0[e] += v[e];
            s1[e] += v[e] * ((z[e] - mu[e]) * rs[e]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < N; ++e) {
    sh[0][threadIdx.x][e] = s0[e];
    sh[1][threadIdx.x][e] = s1[e];
  }
  int half = 1;
  while (2 * half < RG) half *= 2;
  for (; half >= 1; half >>= 1) {
    __syncthreads();
    if (g < half && g + half < RG) {
      const int o = (g + half) * CL + cl;
#pragma unroll
      for (int e = 0; e < N; ++e) {
        sh[0][threadIdx.x][e] += sh[0][o][e];
        sh[1][threadIdx.x][e] += sh[1][o][e];
      }
    }
  }
  if (g == 0 && chunk < chunks) {
    const int c0 = chunk * N;
#pragma unroll
    for (int e = 0; e < N; ++e) {
      b.part[((size_t)(c0 + e) * 2 + 0) * row_blocks + blockIdx.y] = sh[0][cl][e];
      b.part[((size_t)(c0 + e) * 2 + 1) * row_blocks + blockIdx.y] = sh[1][cl][e];
    }
  }
}

// ---------------------------------------------------------------- softmax cross-entropy
constexpr int CE_REG = 8;  // classes per lane kept in registers (up to 512 classes)
// One workgroup; wave w handles rows w, w + 16, ...  Row losses go to LDS and
// one thread adds them in row order.
template <typename T>
__global__ __launch_bounds__(1024) void k_softmax_ce(CeArgs a) {
  __shared__ double row_loss[1024];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const T* Z = (const T*)a.z;
  T* DZ = (T*)a.dz;
  if (a.classes <= 64 * CE_REG) {
    // each lane keeps its logits (classes lane, lane + 64, ...) and their
    // exponentials in registers, and a wave takes two rows at once: the same
    // operations in the same order as the loop below, without re-reading or
    // re-exponentiating
    for (int r0 = wave; r0 < a.n; r0 += 32) {
      double v[2][CE_REG], e[2][CE_REG], mx[2], se[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = r0 + 16 * h;
        mx[h] = -INFINITY;
#pragma unroll
        for (int k = 0; k < CE_REG; ++k) {
          const int c = lane + 64 * k;
          v[h][k] = (r < a.n && c < a.classes) ? ldd(Z + (size_t)r * a.ldz + c) : -INFINITY;
          mx[h] = fmax(mx[h], v[h][k]);
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        mx[h] = wave_max(mx[h]);
        se[h] = 0.0;
#pragma unroll
        for (int k = 0; k < CE_REG; ++k) {
          e[h][k] = lane + 64 * k < a.classes ? exp(v[h][k] - mx[h]) : 0.0;
          se[h] += e[h][k];
        }
        se[h] = wave_sum(se[h]);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = r0 + 16 * h;
        if (r >= a.n) break;
        const int lab = a.labels[r];
        const bool lab_ok = lab >= 0 && lab < a.classes;  // out-of-range label: NaN, no read
        if (lane == 0 && r < 1024)
          row_loss[r] = lab_ok ? -((ldd(Z + (size_t)r * a.ldz + lab) - mx[h]) - log(se[h])) : NAN;
        if (DZ) {
#pragma unroll
          for (int k = 0; k < CE_REG; ++k) {
            const int c = lane + 64 * k;
            if (c >= a.classes) break;
            double p = e[h][k] / se[h];
            if (c == lab) p -= 1.0;
            std_(DZ + (size_t)r * a.lddz + c, lab_ok ? p * a.inv_N : NAN);
          }
        }
      }
    }
    __syncthreads();
    if (threadIdx.x == 0 && a.loss) {
      double s = 0.0;
      for (int r = 0; r < a.n && r < 1024; ++r) s += row_loss[r];
      *a.loss = (float)(s * a.inv_N);
    }
    return;
  }
  for (int r = wave; r < a.n; r += 16) {
    const T* z = Z + (size_t)r * a.ldz;
    double mx = -INFINITY;
    for (int c = lane; c < a.classes; c += 64) mx = fmax(mx, ldd(z + c));
    mx = wave_max(mx);
    double se = 0.0;
    for (int c = lane; c < a.classes; c += 64) se += exp(ldd(z + c) - mx);
    se = wave_sum(se);
    const int lab = a.labels[r];
    const bool lab_ok = lab >= 0 && lab < a.classes;  // out-of-range label: NaN, no read
    if (lane == 0 && r < 1024) row_loss[r] = lab_ok ? -((ldd(z + lab) - mx) - log(se)) : NAN;
    if (DZ) {
      for (int c = lane; c < a.classes; c += 64) {
        double p = exp(ldd(z + c) - mx) / se;
        if (c == lab) p -= 1.0;
        std_(DZ + (size_t)r * a.lddz + c, lab_ok ? p * a.inv_N : NAN);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && a.loss) {
    double s = 0.0;
    for (int r = 0; r < a.n && r < 1024; ++r) s += row_loss[r];
    *a.loss = (float)(s * a.inv_N);
  }
}

hipError_t launch_softmax_ce(int dtype, const CeArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  double cb = (double)a.n * a.classes * (dtype == DT_BF16 ? 2 : 4) * (a.dz ? 2 : 1);
  if (dtype == DT_BF16) XP_LAUNCH("k_softmax_ce<bf16>", cb, k_softmax_ce<bf16_t>, dim3(1), dim3(1024), 0, s, a);
  else XP_LAUNCH("k_softmax_ce<f32>", cb, k_softmax_ce<float>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}


// ============================================================================
// launchers: vectorised path when the views allow 16-byte accesses
// ============================================================================
template <typename T>
static bool fits32(int64_t rows, int C) { return rows * (int64_t)(C / VT<T>::N) < (int64_t)1 << 31; }

template <typename T>
static hipError_t colreduce_t(const ColArgs& a, hipStream_t s) {
  if (fits32<T>(a.M, a.C) && vec_ok<T>(a.C, {{a.a, a.lda}, {a.z, a.ldz}}))
    return colreduce_v<T>(a, s);
  return launch_colreduce_s(sizeof(T) == 2 ? DT_BF16 : DT_F32, a, s);
}
hipError_t launch_colreduce(int dtype, const ColArgs& a, hipStream_t s) {
  if (a.C <= 0 || a.M <= 0) return hipSuccess;
  return dtype == DT_BF16 ? colreduce_t<bf16_t>(a, s) : colreduce_t<float>(a, s);
}

// CHUNK_BYTES: algorithmic bytes moved per 16-byte chunk of the view
#define XP_VEC_LAUNCH(KERNEL, items, CHUNK_BYTES, ...)                                  \
  do {                                                                                   \
    if (dtype == DT_BF16)                                                                \
      XP_LAUNCH(#KERNEL "<bf16>", (double)(items) * (CHUNK_BYTES), KERNEL<bf16_t>,       \
                dim3(grid_for(items)), dim3(256), 0, s, __VA_ARGS__);                    \
    else                                                                                 \
      XP_LAUNCH(#KERNEL "<f32>", (double)(items) * (CHUNK_BYTES), KERNEL<float>,         \
                dim3(grid_for(items)), dim3(256), 0, s, __VA_ARGS__);                    \
    return hipGetLastError();                                                            \
  } while (0)

static bool vec_dt(int dtype, int64_t rows, int C, std::initializer_list<std::pair<const void*, int>> v) {
  return dtype == DT_BF16 ? (fits32<bf16_t>(rows, C) && vec_ok<bf16_t>(C, v))
                          : (fits32<float>(rows, C) && vec_ok<float>(C, v));
}
static int vn(int dtype) { return dtype == DT_BF16 ? 8 : 4; }

// rows per trip of the row kernels (and per thread of their grids); BN
// backward at 4 rather than 2: 7.2 -> 6.3 us (C = 64) and 8.5 -> 6.5 us
// (C = 96) over 32 x 35 x 35 pixels
constexpr int BN_APPLY_U = 4, BN_BWD_U = 4;

hipError_t launch_bn_apply(int dtype, const BnApplyArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  if (a.nseg > 0) {
    // several BNs in one launch: the 16-byte chunk path only, no residual
    const int N = vn(dtype);
    bool ok = a.nseg <= BN_APPLY_SEGS && !a.res && vec_dt(dtype, a.M, a.C, {{a.z, a.ldz}});
    for (int q = 0; ok && q < a.nseg; ++q)
      ok = a.seg_c0[q] % N == 0 && a.seg_c1[q] % N == 0 && a.seg_c0[q] < a.seg_c1[q] &&
           a.seg_c1[q] <= a.C && vec_dt(dtype, a.M, a.seg_c1[q] - a.seg_c0[q], {{a.seg_y[q], a.seg_ldy[q]}});
    if (!ok) return hipErrorInvalidValue;
  }
  if (a.nseg > 0 || vec_dt(dtype, a.M, a.C, {{a.z, a.ldz}, {a.res, a.ldres}, {a.y, a.ldy}})) {
    const int N = vn(dtype);
    const dim3 grid = row_grid(a.M, a.C, N, BN_APPLY_U);
    const double bytes = (double)a.M * a.C * (dtype == DT_BF16 ? 2 : 4) * (a.res ? 3 : 2);
    if (dtype == DT_BF16)
      XP_LAUNCH("k_bn_apply_v<bf16>", bytes, (k_bn_apply_v<bf16_t, BN_APPLY_U>), grid, dim3(256), 0, s, a);
    else
      XP_LAUNCH("k_bn_apply_v<f32>", bytes, (k_bn_apply_v<float, BN_APPLY_U>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  return launch_bn_apply_s(dtype, a, s);
}

hipError_t launch_bn_bwd(int dtype, const BnBwdArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, a.M, a.C, {{a.g, a.ldg}, {a.z, a.ldz}, {a.dz, a.lddz}, {a.dzmask, a.ldzm},
                               {a.dres, a.lddres}, {a.resmask, a.ldrm}})) {
    const int N = vn(dtype);
    const dim3 grid = row_grid(a.M, a.C, N, BN_BWD_U);
    const int tensors = 3 + (a.dzmask ? 1 : 0) + (a.dz_accumulate ? 1 : 0) +
                        (a.dres ? 1 + (a.resmask ? 1 : 0) + (a.res_accumulate ? 1 : 0) : 0);
    const double bytes = (double)a.M * a.C * (dtype == DT_BF16 ? 2 : 4) * tensors;
    if (dtype == DT_BF16)
      XP_LAUNCH("k_bn_bwd_v<bf16>", bytes, (k_bn_bwd_v<bf16_t, BN_BWD_U>), grid, dim3(256), 0, s, a);
    else
      XP_LAUNCH("k_bn_bwd_v<f32>", bytes, (k_bn_bwd_v<float, BN_BWD_U>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  return launch_bn_bwd_s(dtype, a, s);
}

hipError_t launch_elementwise(int dtype, const EltArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, a.M, a.C, {{a.a, a.lda}, {a.b, a.ldb}, {a.mask, a.ldm}, {a.y, a.ldy}}))
    XP_VEC_LAUNCH(k_elt_v, (int64_t)a.M * (a.C / vn(dtype)), vn(dtype) * (dtype == DT_BF16 ? 2 : 4) * (2 + (a.b ? 1 : 0) + (a.mask ? 1 : 0) + (a.accumulate ? 1 : 0)), a);
  return launch_elementwise_s(dtype, a, s);
}

hipError_t launch_maxpool_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int64_t rows = (int64_t)a.nb * (a.H / 2) * (a.W / 2);
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, (int64_t)a.nb * a.H * a.W, a.C, {{a.x, a.ldx}, {a.out, a.ldo}}))
    XP_VEC_LAUNCH(k_maxpool_fwd_v, rows * (a.C / vn(dtype)), vn(dtype) * (dtype == DT_BF16 ? 2 : 4) * 5, a);
  return launch_maxpool_fwd_s(dtype, a, s);
}

hipError_t launch_maxpool_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int64_t rows = (int64_t)a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, rows, a.C, {{a.x, a.ldx}, {a.dy, a.lddy}, {a.mask, a.ldm}, {a.out, a.ldo}}))
    XP_VEC_LAUNCH(k_maxpool_bwd_v, rows * (a.C / vn(dtype)), vn(dtype) * (dtype == DT_BF16 ? 2 : 4) * (2.25 + (a.mask ? 1 : 0) + (a.accumulate ? 1 : 0)), a);
  return launch_maxpool_bwd_s(dtype, a, s);
}

static int avg_blocks(const PoolArgs& a, int n) {
  return ceil_div(a.nb * a.H * ceil_div(a.W, AVG_SEG) * (a.C / n), 256);
}

hipError_t launch_avgpool_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int64_t rows = (int64_t)a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, rows, a.C, {{a.x, a.ldx}, {a.mask, a.ldm}, {a.out, a.ldo}})) {
    const int blocks = avg_blocks(a, vn(dtype));
    if (dtype == DT_BF16)
      XP_LAUNCH("k_avgpool3_v<bf16>", (double)rows * a.C * 2 * ((a.accumulate ? 3 : 2) + (a.mask ? 1 : 0)), k_avgpool3_v<bf16_t>,
                dim3(blocks), dim3(256), 0, s, a, (const bf16_t*)a.x, a.ldx);
    else
      XP_LAUNCH("k_avgpool3_v<f32>", (double)rows * a.C * 4 * ((a.accumulate ? 3 : 2) + (a.mask ? 1 : 0)), k_avgpool3_v<float>,
                dim3(blocks), dim3(256), 0, s, a, (const float*)a.x, a.ldx);
    return hipGetLastError();
  }
  return launch_avgpool_fwd_s(dtype, a, s);
}

hipError_t launch_avgpool_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int64_t rows = (int64_t)a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, rows, a.C, {{a.dy, a.lddy}, {a.mask, a.ldm}, {a.out, a.ldo}})) {
    const int blocks = avg_blocks(a, vn(dtype));
    if (dtype == DT_BF16)
      XP_LAUNCH("k_avgpool3_v<bf16>", (double)rows * a.C * 2 * ((a.accumulate ? 3 : 2) + (a.mask ? 1 : 0)), k_avgpool3_v<bf16_t>,
                dim3(blocks), dim3(256), 0, s, a, (const bf16_t*)a.dy, a.lddy);
    else
      XP_LAUNCH("k_avgpool3_v<f32>", (double)rows * a.C * 4 * ((a.accumulate ? 3 : 2) + (a.mask ? 1 : 0)), k_avgpool3_v<float>,
                dim3(blocks), dim3(256), 0, s, a, (const float*)a.dy, a.lddy);
    return hipGetLastError();
  }
  return launch_avgpool_bwd_s(dtype, a, s);
}

// pixel splits of the GAP partial sums: about 1024 workgroups, >= ~4 pixels per thread
static int gap_splits(int nb, int HW, int C, int n) {
  const int chunks = C / n;
  const int CL = chunks < 256 ? chunks : 256;
  const int RG = 256 / CL;
  int want = ceil_div(1024, nb * ceil_div(chunks, CL));
  const int maxs = ceil_div(HW, RG * 4);
  if (want > maxs) want = maxs;
  if (want > 64) want = 64;
  return want < 1 ? 1 : want;
}
size_t gap_partial_bytes(int nb, int H, int W, int C) {
  return (size_t)nb * 64 * C * sizeof(double);
}

hipError_t launch_gap_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  if (a.nb <= 0 || a.C <= 0) return hipSuccess;
  if (a.part && vec_dt(dtype, (int64_t)a.nb * a.H * a.W, a.C, {{a.x, a.ldx}, {a.out, a.ldo}})) {
    const int chunks = a.C / vn(dtype);
    const int CL = chunks < 256 ? chunks : 256;
    const int colblocks = ceil_div(chunks, CL);
    const int splits = gap_splits(a.nb, a.H * a.W, a.C, vn(dtype));
    dim3 grid(splits, a.nb, colblocks);
    const double gb = (double)a.nb * a.H * a.W * a.C * (dtype == DT_BF16 ? 2 : 4);
    const double fb = (double)a.nb * splits * a.C * 8;
    const int fblocks = ceil_div(a.nb * chunks, 4);
    if (dtype == DT_BF16) {
      XP_LAUNCH("k_gap_part_v<bf16>", gb, k_gap_part_v<bf16_t>, grid, dim3(256), 0, s, a, splits);
      XP_LAUNCH("k_gap_fin_v<bf16>", fb, k_gap_fin_v<bf16_t>, dim3(fblocks), dim3(256), 0, s, a, splits);
    } else {
      XP_LAUNCH("k_gap_part_v<f32>", gb, k_gap_part_v<float>, grid, dim3(256), 0, s, a, splits);
      XP_LAUNCH("k_gap_fin_v<f32>", fb, k_gap_fin_v<float>, dim3(fblocks), dim3(256), 0, s, a, splits);
    }
    return hipGetLastError();
  }
  return launch_gap_fwd_s(dtype, a, s);
}

int gap_bn_max_row_blocks() { return COL_MAX_ROW_BLOCKS_V; }

hipError_t launch_gap_bwd_bn(int dtype, const PoolArgs& a, const GapBnArgs& b, hipStream_t s,
                             int* row_blocks) {
  if (row_blocks) *row_blocks = 0;
  const int64_t rows = (int64_t)a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  const int N = vn(dtype);
  bool ok = b.part && b.bn_nseg >= 1 && b.bn_nseg <= CONV_BN_SEGS &&
            vec_dt(dtype, rows, a.C, {{a.dy, a.lddy}, {a.mask, a.ldm}, {a.out, a.ldo}});
  for (int k = 0; ok && k < b.bn_nseg; ++k)
    ok = b.bn_c0[k] % N == 0 && b.bn_c1[k] % N == 0 && b.bn_c0[k] < b.bn_c1[k] && b.bn_c1[k] <= a.C &&
         vec_dt(dtype, rows, a.C, {{b.bn_z[k], b.ld_bnz[k]}});
  if (!ok) return hipErrorInvalidValue;
  const int rb = col_row_blocks_v((int)rows, a.C, N);
  const int chunks = a.C / N, CL = chunks < 256 ? chunks : 256;
  const dim3 grid(ceil_div(chunks, CL), rb);
  const double bytes = (double)rows * a.C * (dtype == DT_BF16 ? 2 : 4) * (2 + (a.mask ? 1 : 0) + (a.accumulate ? 1 : 0));
  if (dtype == DT_BF16)
    XP_LAUNCH("k_gap_bwd_bn_v<bf16>", bytes, k_gap_bwd_bn_v<bf16_t>, grid, dim3(256), 0, s, a, b, rb);
  else
    XP_LAUNCH("k_gap_bwd_bn_v<f32>", bytes, k_gap_bwd_bn_v<float>, grid, dim3(256), 0, s, a, b, rb);
  if (row_blocks) *row_blocks = rb;
  return hipGetLastError();
}

hipError_t launch_gap_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int64_t rows = (int64_t)a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (vec_dt(dtype, rows, a.C, {{a.dy, a.lddy}, {a.mask, a.ldm}, {a.out, a.ldo}}))
    XP_VEC_LAUNCH(k_gap_bwd_v, rows * (a.C / vn(dtype)), vn(dtype) * (dtype == DT_BF16 ? 2 : 4) * (1 + (a.mask ? 1 : 0) + (a.accumulate ? 1 : 0)), a);
  return launch_gap_bwd_s(dtype, a, s);
}

}  // namespace xp
