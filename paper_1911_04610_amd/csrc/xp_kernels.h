// Host-side interface of the libxpipe kernels: argument blocks and launchers.
// Activation tensors are NHWC views: element (row m, channel c) of a view is
// at ptr[m * ld + c], with m = (n * H + h) * W + w and ptr already offset to
// the view's first channel.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xp {

typedef uint16_t bf16_t;

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

// Optional per-launch observer (kernel timing).  Every launch goes through
// XP_LAUNCH, which calls before() / after(name, work) around it when a hook is
// installed for the calling thread.  work = algorithmic flops for GEMM
// kernels, algorithmic bytes for the others.
struct LaunchHook {
  virtual void before() = 0;
  virtual void after(const char* name, double work) = 0;
  virtual ~LaunchHook() {}
};
extern thread_local LaunchHook* g_hook;

#define XP_LAUNCH(NAME, WORK, KERNEL, GRID, BLOCK, SHM, STREAM, ...)   \
  do {                                                                  \
    if (::xp::g_hook) ::xp::g_hook->before();                           \
    hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHM, STREAM, __VA_ARGS__);  \
    if (::xp::g_hook) ::xp::g_hook->after(NAME, WORK);                  \
  } while (0)

// ---------------------------------------------------------------- prediction / Adam
struct PredCoef {
  double coef;      // s * lr (0 for the identity)
  double c1, c2;    // first / second moment scale (bias correction), 0 for the identity
  double eps;
  int kind;         // PRED_DIR_*: which direction the moments form
};
// directions of the prediction: Eq. 3 (eps inside the root), Adam's own
// (eps after the root), the smoothed gradient alone (first moment times c1)
enum { PRED_DIR_EQ3 = 0, PRED_DIR_ADAM = 1, PRED_DIR_SMOOTHED = 2 };

struct AdamCoef {
  double lr, beta1, beta2, one_m_beta1, one_m_beta2;
  double bc1, bc2;  // 1 / (1 - beta^t) for this update
  double eps;
};

// update rules besides Adam (the prediction keeps reading Adam moments)
constexpr int RULE_MOMENTUM_SGD = 1;
constexpr int RULE_RMSPROP = 2;
struct RuleCoef {
  double lr, mu, wd;                        // step size, momentum, weight decay
  double alpha, one_m_alpha, eps;           // RMSProp squared average and its eps
  double beta1, beta2, one_m_beta1, one_m_beta2;  // the prediction's Adam moments
};

hipError_t launch_predict(const float* W, const float* m, const float* v, float* out,
                          bf16_t* out_bf, int64_t n, const PredCoef& c, hipStream_t s);
hipError_t launch_rule(int rule, float* W, float* B, float* Q, float* m, float* v, float* G, int64_t n,
                       const RuleCoef& c, int zero_grad, float* pf, bf16_t* pf_bf, const PredCoef& cf,
                       float* pb, bf16_t* pb_bf, const PredCoef& cb, hipStream_t s);
hipError_t launch_adam(float* W, float* m, float* v, float* G, int64_t n, const AdamCoef& a,
                       int zero_grad, float* pf, bf16_t* pf_bf, const PredCoef& cf, float* pb,
                       bf16_t* pb_bf, const PredCoef& cb, hipStream_t s);

// ---------------------------------------------------------------- weight gather
// Copies nseg blocks of elements (storage dtype) back to back into dst: the
// weights of sibling layers that share one GEMM launch.
constexpr int GATHER_MAX_SEGS = 4;
// copies src[j] -> dst[j] (count[j] elements) for j < nseg, one launch
constexpr int GATHER_BATCH = 16;
struct GatherArgs {
  int nseg;
  const void* src[GATHER_BATCH];
  void* dst[GATHER_BATCH];
  int64_t count[GATHER_BATCH];
};
hipError_t launch_gather(int dtype, const GatherArgs& a, hipStream_t s);

// ---------------------------------------------------------------- GEMM engine
// Forward-type implicit GEMM: y[m][n] = act(sum_{r,s,c} x[pix(m) + (r-pad, s-pad)][c] *
// w[n][r][s][c] + bias[n]) over an nb x H x W image batch (stride 1, zero padding).
// Serves conv forward, linear forward (H = W = R = S = 1) and the data gradient
// (x = output gradient, w = flipped / transposed weights).
constexpr int CONV_BN_SEGS = 4;
struct ConvArgs {
  const void* x;
  int ldx;
  const void* w;        // [N][R][S][C] contiguous, storage dtype
  void* y;
  int ldy;
  const float* bias;    // [N] or null
  const void* mask;     // optional view: y *= (mask > 0)
  int ldm;
  int nb, H, W, C, N, R, S, pad;  // pad: rows (and columns when padw is unset)
  int relu;             // apply max(., 0) before storing
  int accumulate;       // y = y + result (after mask)
  double* stat_part;    // optional: per row tile, column sums of the stored y and of its
                        // squares, at stat_part[(n * 2 + {0,1}) * row_tiles + tile]
  // optional (bf16): columns [bn_c0[k], bn_c1[k]) of the stored y are the
  // output gradient g of batch norm k (k < bn_nseg), whose input is z (view
  // bn_z[k], ld_bnz[k]) with batch mean / rstd bn_mean[k] / bn_rstd[k] (all
  // three from the norm's first column on); per row tile, the column sums of
  // g and of g (z - mean) rstd, at bn_part[(n * 2 + {0,1}) * row_tiles + tile]
  // (the BN backward's partials; columns outside every range get zeros).
  // bn_z[k] == nullptr: a bias's columns, the sums of g alone (second sum 0)
  double* bn_part;
  int bn_nseg;
  int bn_c0[CONV_BN_SEGS], bn_c1[CONV_BN_SEGS];
  const void* bn_z[CONV_BN_SEGS];
  int ld_bnz[CONV_BN_SEGS];
  const double* bn_mean[CONV_BN_SEGS];
  const double* bn_rstd[CONV_BN_SEGS];
  // general grid (Ho > 0: strided, or unpadded): the rows are an Ho x Wo grid
  // per image, stride >= 1.
  // tr = 0: forward, row (ho, wo) reads x at (ho*stride + r - pad, wo*stride + q - padw);
  // tr = 1: data gradient, x is the output gradient (H x W), the rows the
  // input grid, and row (h, w) reads x at ((h + pad - r) / stride, ...) where
  // stride divides h + pad - r, with the weights transposed but not flipped
  int stride, Ho, Wo, tr;
  int padw;             // column padding
};

// Weight gradient: part[split][n][k] = sum_{m in split} dz[m][n] * x~[m][k],
// k = (r, s, c); then grad[n][k] += sum over splits (fixed order).
struct WgradArgs {
  const void* dz;
  int lddz;
  const void* x;
  int ldx;
  void* part;           // workspace: splits x N x K partial sums (fp32 or fp64)
  float* grad;          // [N][K] fp32 accumulator
  int nb, H, W, C, N, R, S, pad;
  int splits;
  // general grid (Ho > 0): dz has Ho x Wo pixels per image, pixel (ho, wo)
  // pairs with x at (ho*stride + r - pad, wo*stride + q - padw)
  int stride, Ho, Wo;
  int padw;             // column padding
  // optional (nseg > 0): the N rows go to nseg accumulators in order, rows
  // [seg_row0[j], seg_row0[j + 1]) to seg_grad[j] (seg_row0[0] = 0, seg_row0[nseg] = N)
  int nseg;
  int seg_row0[GATHER_MAX_SEGS + 1];
  float* seg_grad[GATHER_MAX_SEGS];
  // set by the launcher (bf16 chunk path, one split): the tile is added
  // straight into grad (or seg_grad) and no partials are written
  int direct;
};

// Work plan of one GEMM launch (tile shape picked on the host).
// grid_rows (optional) receives the number of row tiles of the launch
hipError_t launch_conv_gemm(int dtype, const ConvArgs& a, hipStream_t s, int* grid_rows = nullptr);
// row tiles the forward-type GEMM uses for M rows (upper bound over tile choices)
int conv_max_row_tiles(int M);
size_t wgrad_part_bytes(int dtype, int N, int K, int splits);
// pixel splits of the weight gradient (R*S = taps filter positions)
int wgrad_pick_splits(int dtype, int M, int N, int K, int taps);
hipError_t launch_wgrad(int dtype, const WgradArgs& a, hipStream_t s);

// Transposed copies of the convolutions' weights for their data gradients,
// flipped for stride 1, up to FLIP_MAX per launch (grid y = the convolution):
// wd[c][r][s][n] = w[n][R-1-r][S-1-s][c] (flip != 0) or w[n][r][s][c] (flip == 0).
constexpr int FLIP_MAX = 32;
struct FlipSet {
  int n;
  const void* w[FLIP_MAX];
  void* wd[FLIP_MAX];
  int N[FLIP_MAX], R[FLIP_MAX], S[FLIP_MAX], C[FLIP_MAX], flip[FLIP_MAX];
};
hipError_t launch_flip_set(int dtype, const FlipSet& f, hipStream_t s);

// ---------------------------------------------------------------- column reductions
// Per-column sums over the rows of [M][C] views, two-level and fixed-order.
enum ColMode { COL_STATS = 0, COL_BNBWD = 1, COL_BIAS = 2 };
struct ColArgs {
  int mode;
  const void* a;        // STATS: z; BNBWD: g; BIAS: g
  int lda;
  const void* z;        // BNBWD: BN input
  int ldz;
  const double* mean;   // BNBWD
  const double* rstd;   // BNBWD
  int M, C;
  double* partial;      // workspace [C][2][row blocks]
  int row_blocks;
  // finalize outputs
  double* out0;         // STATS: mean; BNBWD: dbeta
  double* out1;         // STATS: rstd; BNBWD: dgamma
  float* grad0;         // BNBWD: grad of gamma; BIAS: grad of bias (accumulated)
  float* grad1;         // BNBWD: grad of beta
  double eps;
};
int col_row_blocks(int M, int C);
size_t col_partial_bytes(int M, int C);
hipError_t launch_colreduce(int dtype, const ColArgs& a, hipStream_t s);
// second level only: sums a.row_blocks partials per column and finalises (a.mode)
hipError_t launch_colfinal(const ColArgs& a, hipStream_t s);

// ---------------------------------------------------------------- element-wise
constexpr int BN_APPLY_SEGS = 4;
struct BnApplyArgs {
  const void* z; int ldz;
  const double* mean; const double* rstd;
  const float* gamma; const float* beta;
  const void* res; int ldres;     // optional residual (added before the ReLU)
  void* y; int ldy;
  int M, C, relu;
  // nseg > 0: the BNs over channel ranges [seg_c0, seg_c1) of z (multiples of
  // the 16-byte chunk; mean / rstd indexed by the channel of z), each with its
  // own output, gamma / beta (from its first channel) and ReLU flag; y, gamma,
  // beta and relu above are unused, and so is res (none)
  int nseg;
  int seg_c0[BN_APPLY_SEGS], seg_c1[BN_APPLY_SEGS];
  void* seg_y[BN_APPLY_SEGS]; int seg_ldy[BN_APPLY_SEGS];
  const float* seg_gamma[BN_APPLY_SEGS]; const float* seg_beta[BN_APPLY_SEGS];
  int seg_relu[BN_APPLY_SEGS];
};
hipError_t launch_bn_apply(int dtype, const BnApplyArgs& a, hipStream_t s);

struct BnBwdArgs {
  const void* g; int ldg;          // gradient at the BN(+add) output, masked
  const void* z; int ldz;
  const double* mean; const double* rstd;
  const double* dbeta; const double* dgamma;
  const float* gamma;
  void* dz; int lddz;              // BN-input gradient
  const void* dzmask; int ldzm;    // optional mask for dz
  int dz_accumulate;
  void* dres; int lddres;          // optional residual-source gradient
  const void* resmask; int ldrm;   // optional mask for dres
  int res_accumulate;
  int M, C;
};
hipError_t launch_bn_bwd(int dtype, const BnBwdArgs& a, hipStream_t s);

// y = relu?(a [+ b]), or mask mode: y = a * (m > 0)
struct EltArgs {
  const void* a; int lda;
  const void* b; int ldb;          // optional second operand (add)
  const void* mask; int ldm;       // optional mask
  void* y; int ldy;
  int M, C, relu, accumulate;
};
hipError_t launch_elementwise(int dtype, const EltArgs& a, hipStream_t s);

struct PoolArgs {
  const void* x; int ldx;          // pool input view
  const void* y; int ldy;          // pool output view (forward result)
  const void* dy; int lddy;        // backward: output gradient
  void* out; int ldo;              // forward: y; backward: dx
  const void* mask; int ldm;       // backward: mask for dx
  int accumulate;
  int nb, H, W, C;                 // input shape
  double* part;                    // GAP forward: workspace, gap_partial_bytes
  int valid;                       // 3x3 stride-2 max pool: no padding
  // 3x3 stride-2 max pool: per output element, the window position r * 3 + q
  // of the first maximum, one byte, at idx[row * ldi + channel]; the forward
  // writes it when given, the backward requires it
  uint8_t* idx; int ldi;
};
size_t gap_partial_bytes(int nb, int H, int W, int C);
hipError_t launch_maxpool_fwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_maxpool_bwd(int dtype, const PoolArgs& a, hipStream_t s);
// 3x3 / stride 2 / padding 1 max pool (padding never chosen; ties to the first
// maximum in row-major window order); the backward takes each window's choice
// from a.idx, which the forward recorded
hipError_t launch_maxpool3s2_fwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_maxpool3s2_bwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_avgpool_fwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_avgpool_bwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_gap_fwd(int dtype, const PoolArgs& a, hipStream_t s);
hipError_t launch_gap_bwd(int dtype, const PoolArgs& a, hipStream_t s);
// GAP backward (a's dy, mask, out, accumulate, shape) that also takes the
// batch-norm backward partials of the norms whose output gradient it
// completes: columns [bn_c0[k], bn_c1[k]) belong to norm k (k < bn_nseg, each
// boundary a multiple of the 16-byte chunk), whose input is z (view bn_z[k],
// ld_bnz[k]) with mean / rstd bn_mean[k] / bn_rstd[k], all from the norm's
// first column on.  Per row block, the column sums of the stored gradient g
// and of g (z - mean) rstd go to part[(c * 2 + {0,1}) * row_blocks + block]
// (zeros outside the norms' columns); *row_blocks receives the block count
// (at most gap_bn_max_row_blocks()).  Vector path only: hipErrorInvalidValue
// when the views are not 16-byte aligned.
struct GapBnArgs {
  double* part;
  int bn_nseg;
  int bn_c0[CONV_BN_SEGS], bn_c1[CONV_BN_SEGS];
  const void* bn_z[CONV_BN_SEGS];
  int ld_bnz[CONV_BN_SEGS];
  const double* bn_mean[CONV_BN_SEGS];
  const double* bn_rstd[CONV_BN_SEGS];
};
hipError_t launch_gap_bwd_bn(int dtype, const PoolArgs& a, const GapBnArgs& b, hipStream_t s,
                             int* row_blocks);
int gap_bn_max_row_blocks();

struct CeArgs {
  const void* z; int ldz;          // logits [n][classes]
  const int32_t* labels;
  int n, classes;
  double inv_N;                    // 1 / mini-batch size
  float* loss;                     // forward: loss share (may be null)
  void* dz; int lddz;              // backward: dlogits (may be null)
};
hipError_t launch_softmax_ce(int dtype, const CeArgs& a, hipStream_t s);

// ---------------------------------------------------------------- measurement probes
hipError_t launch_probe_copy(const void* src, void* dst, int64_t bytes, hipStream_t s);
hipError_t launch_probe_mfma(float* out, int waves, int iters, hipStream_t s);
hipError_t launch_probe_spin(float* p, int i, int iters, int blocks, hipStream_t s);
// measurement probe: n 16-byte vectors read from each of nsrc buffers and
// written to each of ndst buffers
constexpr int STREAM_MAX_SRC = 4, STREAM_MAX_DST = 6;
struct StreamArgs {
  const float* src[STREAM_MAX_SRC];
  float* dst[STREAM_MAX_DST];
  int nsrc, ndst;
  int64_t n;  // 16-byte vectors per buffer
};
hipError_t launch_probe_stream(const StreamArgs& a, hipStream_t s);


}  // namespace xp
