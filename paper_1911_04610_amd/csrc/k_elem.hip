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
size_t col_partial_bytes(int M, int C) {
  return (size_t)row_blocks_for(M, C) * 2 * C * sizeof(double);
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
    a.partial[((size_t)blockIdx.y * 2 + 0) * a.C + col] = t0;
    a.partial[((size_t)blockIdx.y * 2 + 1) * a.C + col] = t1;
  }
}

__global__ __launch_bounds__(256) void k_colfinal(ColArgs a) {
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  if (col >= a.C) return;
  double s0 = 0.0, s1 = 0.0;
  for (int b = 0; b < a.row_blocks; ++b) {
    s0 += a.partial[((size_t)b * 2 + 0) * a.C + col];
    s1 += a.partial[((size_t)b * 2 + 1) * a.C + col];
  }
  if (a.mode == COL_STATS) {
    double mean = s0 / a.M;
    double var = s1 / a.M - mean * mean;
    if (var < 0.0) var = 0.0;
    a.out0[col] = mean;
    a.out1[col] = 1.0 / sqrt(var + a.eps);
  } else if (a.mode == COL_BNBWD) {
    a.out0[col] = s0;  // dbeta
    a.out1[col] = s1;  // dgamma
    a.grad0[col] = (float)((double)a.grad0[col] + s1);
    a.grad1[col] = (float)((double)a.grad1[col] + s0);
  } else {
    a.grad0[col] = (float)((double)a.grad0[col] + s0);
  }
}

template <typename T>
static hipError_t colreduce_go(const ColArgs& a, hipStream_t s) {
  dim3 grid(ceil_div(a.C, 64), a.row_blocks);
  hipLaunchKernelGGL(k_colpart<T>, grid, dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_colfinal, dim3(ceil_div(a.C, 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_colreduce(int dtype, const ColArgs& a, hipStream_t s) {
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
    if (R) v += ldd(R + (size_t)r * a.ldres + col);
    if (a.relu) v = v > 0.0 ? v : 0.0;
    std_(Y + (size_t)r * a.ldy + col, v);
  }
}

hipError_t launch_bn_apply(int dtype, const BnApplyArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(k_bn_apply<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    hipLaunchKernelGGL(k_bn_apply<float>, grid, dim3(256), 0, s, a, rb);
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

hipError_t launch_bn_bwd(int dtype, const BnBwdArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(k_bn_bwd<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    hipLaunchKernelGGL(k_bn_bwd<float>, grid, dim3(256), 0, s, a, rb);
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

hipError_t launch_elementwise(int dtype, const EltArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(a.M, a.C);
  dim3 grid(ceil_div(a.C, 64), rb);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(k_elt<bf16_t>, grid, dim3(256), 0, s, a, rb);
  else
    hipLaunchKernelGGL(k_elt<float>, grid, dim3(256), 0, s, a, rb);
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
static void pool_launch_rows(void (*k)(PoolArgs, int, int), const PoolArgs& a, int rows,
                             hipStream_t s) {
  int rb = row_blocks_for(rows, a.C);
  hipLaunchKernelGGL(k, dim3(ceil_div(a.C, 64), rb), dim3(256), 0, s, a, rows, rb);
}

hipError_t launch_maxpool_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * (a.H / 2) * (a.W / 2);
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_maxpool_fwd<bf16_t>, a, rows, s);
  else pool_launch_rows<float>(k_maxpool_fwd<float>, a, rows, s);
  return hipGetLastError();
}

hipError_t launch_maxpool_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_maxpool_bwd<bf16_t>, a, rows, s);
  else pool_launch_rows<float>(k_maxpool_bwd<float>, a, rows, s);
  return hipGetLastError();
}

template <typename T>
static hipError_t avg_go(const PoolArgs& a, const void* src, int ld_src, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  int rb = row_blocks_for(rows, a.C);
  hipLaunchKernelGGL(k_avgpool3<T>, dim3(ceil_div(a.C, 64), rb), dim3(256), 0, s, a,
                     (const T*)src, ld_src, rows, rb);
  return hipGetLastError();
}

hipError_t launch_avgpool_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  return dtype == DT_BF16 ? avg_go<bf16_t>(a, a.x, a.ldx, s) : avg_go<float>(a, a.x, a.ldx, s);
}

hipError_t launch_avgpool_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  return dtype == DT_BF16 ? avg_go<bf16_t>(a, a.dy, a.lddy, s) : avg_go<float>(a, a.dy, a.lddy, s);
}

hipError_t launch_gap_fwd(int dtype, const PoolArgs& a, hipStream_t s) {
  if (a.nb <= 0 || a.C <= 0) return hipSuccess;
  dim3 grid(ceil_div(a.C, 64), a.nb);
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_gap_fwd<bf16_t>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_gap_fwd<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gap_bwd(int dtype, const PoolArgs& a, hipStream_t s) {
  int rows = a.nb * a.H * a.W;
  if (rows <= 0 || a.C <= 0) return hipSuccess;
  if (dtype == DT_BF16) pool_launch_rows<bf16_t>(k_gap_bwd<bf16_t>, a, rows, s);
  else pool_launch_rows<float>(k_gap_bwd<float>, a, rows, s);
  return hipGetLastError();
}

// ---------------------------------------------------------------- softmax cross-entropy
// One workgroup; wave w handles rows w, w + 16, ...  Row losses go to LDS and
// one thread adds them in row order.
template <typename T>
__global__ __launch_bounds__(1024) void k_softmax_ce(CeArgs a) {
  __shared__ double row_loss[1024];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const T* Z = (const T*)a.z;
  T* DZ = (T*)a.dz;
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
  if (dtype == DT_BF16) hipLaunchKernelGGL(k_softmax_ce<bf16_t>, dim3(1), dim3(1024), 0, s, a);
  else hipLaunchKernelGGL(k_softmax_ce<float>, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

}  // namespace xp
