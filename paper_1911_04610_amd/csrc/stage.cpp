// libxpipe host runtime: stage planning, launch sequencing and the C ABI.
//
// A stage is a layer list (see include/xpipe.h).  At creation the runtime
//   - checks every layer and infers NHWC shapes,
//   - lays out the flat parameter buffer (64-element aligned tensors),
//   - groups layers into fused launches: conv/linear (+ReLU in the epilogue),
//     BN (+residual add) (+ReLU), add (+ReLU), pools, GAP, softmax-CE; a
//     concatenation costs nothing: its inputs are produced straight into
//     channel slices of its buffer,
//   - gives every group output an activation buffer and a gradient buffer in
//     the caller's workspace.  A gradient buffer of a ReLU output holds the
//     gradient of the pre-activation: every producer multiplies by the mask
//     (output > 0) as it writes.
//   - fixes, for each gradient buffer, which producer writes first and which
//     ones add (reverse layer order), so the backward is deterministic.
// Each call then only enqueues kernels on the stage's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <iterator>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/xpipe.h"
#include "xp_kernels.h"

using namespace xp;

namespace {

thread_local std::string g_err;

xpipe_status fail(xpipe_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define XP_HIP(call)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail(XPIPE_EHIP, std::string(#call) + ": " + hipGetErrorString(e_));        \
  } while (0)

constexpr int64_t PARAM_ALIGN = 64;  // elements
constexpr size_t WS_ALIGN = 256;     // bytes
constexpr double BN_EPS = 1e-5;
// launch lanes: the stage's stream plus auxiliary streams on which independent
// branches of the layer graph run concurrently.  Three: on the Inception-A
// step (four branches per module) a fourth lane made the recorded step slower
// (8.24 against 7.88 ms), and so did six or eight lanes (8.8 ms), two (7.97)
// or one (9.64)
constexpr int NLANES = 3;
// lanes a pass may start new chains on.  The backward (recompute, data and
// weight gradients) keeps the GPU busy with two: a third lane there made the
// Inception-A step slower (6.65 against 6.62 ms; one lane: 7.80 ms), while
// the forward, bound by launch latency, loses with fewer than three (two:
// 6.94 ms, one: 7.98 ms)
constexpr int PASS_LANES[2] = {3, 2};

int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

struct Shape {
  int n = 0, H = 0, W = 0, C = 0;
  int64_t rows() const { return (int64_t)n * H * W; }
  int64_t elems() const { return rows() * C; }
};

enum OpKind { OP_GEMM, OP_BN, OP_ELT, OP_MAXPOOL, OP_AVGPOOL, OP_GAP, OP_CONCAT, OP_CE, OP_MAXPOOL3 };

struct Tensor {
  Shape sh;
  int owner = -1;        // owning tensor id for a concat member view, else -1
  int coff = 0;          // channel offset in the owner
  int64_t act_off = -1;  // workspace byte offset of the owner's activation buffer
  int64_t grad_off = -1; // workspace byte offset of the owner's gradient buffer
  bool masked = false;   // values are ReLU outputs
  int consumers = 0;
};

struct Op {
  OpKind kind = OP_ELT;
  int layer = -1;      // primary layer
  int in = -1;         // input tensor
  int in2 = -1;        // residual / second add operand tensor
  int out = -1;        // output tensor (-1 for CE)
  bool relu = false;
  // GEMM
  int cin = 0, cout = 0, k = 1, stride = 1;
  int kw = 1, ph = 0, pw = 0;       // kernel width, row / column zero padding
  bool grid = false;                // output grid differs from the input's (strided or unpadded)
  bool valid = false;               // 3x3 stride-2 max pool without padding
  int64_t w_off = -1, b_off = -1;   // parameter offsets (elements)
  int64_t wd_off = -1;              // workspace bytes: flipped weights for the data gradient
  // GEMM over sibling layers that read the same input (merged launch): their
  // weight tensors (parameter offset, output channels) in output-channel order
  std::vector<std::pair<int64_t, int>> segs;
  int64_t wg_off[2] = {-1, -1};     // workspace bytes: gathered predicted weights per direction
  // 3x3 stride-2 max pool: workspace bytes of the first-maximum positions (one
  // byte per output element), written by the forward that the backward
  // recomputes and read by the pool's backward
  int64_t idx_off = -1;
  // BN
  int64_t g_off = -1, be_off = -1;  // gamma / beta parameter offsets
  int64_t stat_off = -1;            // workspace bytes: mean, rstd, dbeta, dgamma (doubles) ...
  int stat_ld = 0;                  // ... arrays stat_ld doubles apart
  // backward bookkeeping: first producer writes, later ones add
  bool in_acc = false, in2_acc = false;
  // batch-norm statistics computed in the producing GEMM's epilogue
  bool stats = false;          // GEMM: writes mean / rstd of every output column ...
  int64_t stat_block = -1;     // ... to this workspace block ([2][cout] doubles, then dbeta/dgamma)
  bool stats_fused = false;    // BN: statistics come from the producing GEMM
  int stats_from = -1;         // BN: index of that GEMM op
  // bf16: BNs whose output gradients are completed by one GEMM's data
  // gradient (the last of its input's gradient writers) take their backward
  // column sums from that launch's epilogue
  std::vector<std::pair<int, int>> bnb_segs;  // GEMM: (BN op, first input column) each
  int bnb_gemm = -1;           // BN: the GEMM op that computes them ...
  int bnb_c0 = 0;              // ... at this input column of it
  int64_t bnb_part_off = -1;   // GEMM: workspace bytes of those per-row-tile partials
  // bf16: a 1x1 convolution whose input is a 3x3 average pool (padding
  // counted) takes the pool's backward: its output gradient is box-averaged
  // first (the pool is self-adjoint and commutes with the 1x1 contraction),
  // and its data gradient writes the pool input's gradient directly
  int pool_bwd = -1;           // GEMM: the average-pool op
  int pool_by = -1;            // AVGPOOL: the GEMM op that takes its backward
  int64_t box_off = -1;        // GEMM: workspace bytes of the averaged output gradient
  int apply_grp = -1;          // BN: its group of BNs over one merged GEMM's slices
  // launch lanes, per pass (0 forward, 1 backward): the lane this op runs on,
  // the ops (same pass) on other lanes it waits for, and whether later ops on
  // other lanes wait for it
  int lane[2] = {0, 0};
  std::vector<int> waits[2];
  bool record[2] = {false, false};
};

struct ParamT {
  int64_t off, count;
};

struct TimeRec {
  hipEvent_t a, b;
  const char* name;
  double work;
};

struct TimeAgg {
  double ms = 0, work = 0;
  int64_t n = 0;
};

}  // namespace

struct xpipe_stage {
  std::vector<xpipe_layer_desc> layers;
  int mb = 0, T = 1, dtype = DT_F32;
  Shape in_shape;
  hipStream_t stream = nullptr;     // the stream launches go to (swapped while a pass records or a forward runs on fwd_stream)
  hipStream_t own_stream = nullptr; // the stage's stream as created
  float *W = nullptr, *m = nullptr, *v = nullptr, *grad = nullptr;
  float *wpf = nullptr, *wpb = nullptr;
  // workspace: ws holds the running pass's activations, gradients and
  // scratch; wws the weight copies derived from the predictions (bf16
  // shadows, gathered and flipped weights), written only by the prediction
  // and update calls.  Both are the caller's workspace, except while a
  // forward runs on its own stream (fwd_stream): then ws is fwd_ws.
  char* ws = nullptr;
  char* wws = nullptr;
  size_t ws_bytes = 0;
  size_t ws_need = 0;  // the plan's workspace size (xpipe_stage_query)
  hipStream_t fwd_stream = nullptr;
  char* fwd_ws = nullptr;
  hipEvent_t pred_ev = nullptr;  // stage stream: the last write of the forward prediction
  hipEvent_t fwd_ev = nullptr;   // fwd_stream: the last forward
  bool fwd_pending = false;      // a forward was enqueued on fwd_stream since the stage stream last waited
  int64_t P = 0;
  std::vector<ParamT> params;
  std::vector<Tensor> tensors;  // [0] = stage input
  std::vector<Op> ops;
  std::vector<int> bnb_nrb;     // per GEMM op with bnb_segs: row tiles of its last data-gradient launch
  int out_tensor = -1;          // stage output tensor (logits for a loss stage)
  bool has_loss = false;
  int classes = 0;
  int64_t bf_f_off = -1, bf_b_off = -1;  // bf16 shadows of the predictions
  int64_t colpart_off[NLANES] = {}, wpart_off[NLANES] = {};  // per-lane scratch
  hipStream_t lane_stream[NLANES] = {};  // [0] = the stage's stream
  std::vector<hipEvent_t> op_ev[2];      // per op, per pass
  hipEvent_t fork_ev = nullptr, join_ev[NLANES] = {};
  // call-order state
  bool pred_valid[2] = {false, false};
  bool wd_valid = false;
  int64_t bwd_since_step = 0;
  // timing: hipEvents around every launch, aggregated per kernel
  struct Hook : xp::LaunchHook {
    xpipe_stage* st = nullptr;
    hipEvent_t a = nullptr;
    void before() override;
    void after(const char* name, double work) override;
  } hook;
  bool timing = false;
  // a stage of xpipe_stage_create_static: one launch lane (no auxiliary
  // streams or events), no recorded passes, workspace in the static array of
  // device static_dev
  bool one_lane = false;
  int static_dev = -1;
  // recorded passes: each distinct (pass, caller pointers) is captured once
  // into a HIP graph on cap_stream and replayed on the stage's stream
  struct PassGraph {
    int kind;                // 0 forward, 1 backward
    const void* ptr[5];      // the call's pointers
    hipGraphExec_t exec;
    uint64_t used;           // last use, for eviction
  };
  bool graphs = true;
  bool capturing = false;  // a pass is being recorded on cap_stream
  std::vector<int> rec_order[2];  // op order while recording (see Plan)
  std::vector<std::vector<int>> apply_groups;
  hipStream_t cap_stream = nullptr;
  std::vector<PassGraph> pass_graphs;
  uint64_t graph_clock = 0;
  std::vector<TimeRec> pending;
  std::vector<hipEvent_t> pool;
  std::map<std::string, TimeAgg> agg;

  size_t esz() const { return dtype == DT_BF16 ? 2 : 4; }
};

namespace {

// ============================================================================
// planning
// ============================================================================
struct Plan {
  std::vector<ParamT> params;
  std::vector<Tensor> tensors;
  std::vector<Op> ops;
  int out_tensor = -1;
  bool has_loss = false;
  int classes = 0;
  int64_t P = 0;
  size_t ws = 0;
  int64_t bf_f_off = -1, bf_b_off = -1, colpart_off[NLANES] = {}, wpart_off[NLANES] = {};
  // per pass, the order in which a recorded pass captures its ops: a
  // topological order of the lane plan that takes the lanes in turn, so the
  // graph's launches interleave the independent branches
  std::vector<int> rec_order[2];
  std::vector<std::vector<int>> apply_groups;  // BN ops applied by one launch (see Op)
};

// Channel range a tensor occupies in its buffer: (buffer tensor, first, end).
struct Region {
  int base, c0, c1;
};
Region region_of(const Plan& p, int t) {
  const Tensor& tt = p.tensors[t];
  const int b = tt.owner >= 0 ? tt.owner : t;
  return Region{b, tt.coff, tt.coff + tt.sh.C};
}
bool overlap(const Region& a, const Region& b) {
  return a.base == b.base && a.c0 < b.c1 && b.c0 < a.c1;
}

// Assigns every op a lane per pass and the cross-lane waits that keep the
// launch order's data dependencies.  Forward: an op depends on the ops that
// wrote what it reads.  Backward (ops in reverse): an op depends on the ops
// that wrote the gradient it reads and on the earlier writers of the gradient
// it writes (the fixed accumulation order).  An op continues the lane of a
// dependency that is still that lane's last op, else takes the next lane in
// turn; waits on same-lane dependencies are implied by stream order.
void plan_lanes(Plan& p) {
  const int n = (int)p.ops.size();
  auto writes_fwd = [&](int j) -> int { return p.ops[j].kind == OP_CE ? -1 : p.ops[j].out; };
  for (int pass = 0; pass < 2; ++pass) {
    std::vector<std::vector<int>> deps(n);
    for (int i = 0; i < n; ++i) {
      const Op& op = p.ops[i];
      if (op.kind == OP_CONCAT) continue;
      if (pass == 0) {
        for (int r : {op.in, op.in2}) {
          if (r <= 0) continue;  // the stage input is ready before the pass
          const Region rr = region_of(p, r);
          for (int j = 0; j < i; ++j) {
            const int w = writes_fwd(j);
            if (w >= 0 && p.ops[j].kind != OP_CONCAT && overlap(region_of(p, w), rr))
              deps[i].push_back(j);
          }
        }
      } else {
        // backward order is n-1 .. 0: "earlier" means a larger index
        auto grad_writes = [&](int j, const Region& rr) {
          const Op& o = p.ops[j];
          if (o.kind == OP_CONCAT) return false;
          // (tensor 0 is the stage input: its gradient is the caller's dx)
          for (int t : {o.in, o.in2})
            if (t >= 0 && overlap(region_of(p, t), rr)) return true;
          return false;
        };
        std::vector<Region> rs;
        if (op.kind != OP_CE) rs.push_back(region_of(p, op.out));
        for (int t : {op.in, op.in2})
          if (t >= 0) rs.push_back(region_of(p, t));
        for (int j = n - 1; j > i; --j)
          for (const Region& rr : rs)
            if (grad_writes(j, rr)) {
              deps[i].push_back(j);
              break;
            }
      }
    }
    auto qpos = [&](int i) { return pass == 0 ? i : n - 1 - i; };
    std::vector<int> tail(NLANES, -1), tail_q(NLANES, -1);
    // per lane: the pass position up to which each lane's ops are known to
    // have completed (lane order and the waits so far); per op, that vector
    // when it was placed
    std::vector<std::array<int, NLANES>> vc(n);
    std::array<int, NLANES> lane_vc[NLANES];
    for (int l = 0; l < NLANES; ++l) lane_vc[l].fill(-1);
    for (int q = 0; q < n; ++q) {
      const int i = pass == 0 ? q : n - 1 - q;
      Op& op = p.ops[i];
      op.waits[pass].clear();
      if (op.kind == OP_CONCAT) continue;
      // continue the chain of the most recent dependency that ends its lane,
      // else start on the lane that has been idle longest
      int lane = -1, best_q = -1;
      for (int j : deps[i]) {
        const int l = p.ops[j].lane[pass];
        if (tail[l] == j && tail_q[l] > best_q) {
          lane = l;
          best_q = tail_q[l];
        }
      }
      if (lane < 0) {
        lane = 0;
        for (int l = 1; l < PASS_LANES[pass]; ++l)
          if (tail_q[l] < tail_q[lane]) lane = l;
      }
      op.lane[pass] = lane;
      tail[lane] = i;
      tail_q[lane] = q;
      // waits for ops on other lanes, skipping those already covered by lane
      // order and earlier waits (latest first: a wait for a later op of a
      // lane covers its earlier ones); the graph gets no redundant edges
      std::vector<int> ds = deps[i];
      std::sort(ds.begin(), ds.end(), [&](int a, int b) { return qpos(a) > qpos(b); });
      for (int j : ds) {
        const int m = p.ops[j].lane[pass];
        if (m == lane || lane_vc[lane][m] >= qpos(j)) continue;
        op.waits[pass].push_back(j);
        p.ops[j].record[pass] = true;
        for (int l = 0; l < NLANES; ++l) lane_vc[lane][l] = std::max(lane_vc[lane][l], vc[j][l]);
      }
      lane_vc[lane][lane] = q;
      vc[i] = lane_vc[lane];
    }
    // recording order: an op is ready once the previous op of its lane (in
    // pass order) and the ops it waits for are placed; among ready ops take
    // the one with the longest path to the end of the pass (GEMM ops weigh 3
    // forward, 6 backward, the others 1), then pass order.  The graph's nodes
    // are dispatched in this order when several are ready: on the Inception-A
    // step this took 7.77 -> 7.57 ms against taking the lane placed least
    // recently (7.85 ms in plain pass order); other weights gave the same
    std::vector<int> seq;  // pass order without concats
    for (int q = 0; q < n; ++q) {
      const int i = pass == 0 ? q : n - 1 - q;
      if (p.ops[i].kind != OP_CONCAT) seq.push_back(i);
    }
    std::vector<int> prev(n, -1), last(NLANES, -1);
    for (int i : seq) {
      prev[i] = last[p.ops[i].lane[pass]];
      last[p.ops[i].lane[pass]] = i;
    }
    std::vector<double> level(n, 0.0);  // longest weighted path to the pass end
    {
      std::vector<std::vector<int>> succ(n);
      for (int i : seq) {
        if (prev[i] >= 0) succ[prev[i]].push_back(i);
        for (int j : p.ops[i].waits[pass]) succ[j].push_back(i);
      }
      for (int q = (int)seq.size() - 1; q >= 0; --q) {
        const int i = seq[q];
        double m = 0.0;
        for (int k : succ[i]) m = std::max(m, level[k]);
        level[i] = (p.ops[i].kind == OP_GEMM ? (pass == 1 ? 6.0 : 3.0) : 1.0) + m;
      }
    }
    std::vector<char> placed(n, 0);
    std::vector<int>& order = p.rec_order[pass];
    order.clear();
    while (order.size() < seq.size()) {
      int pick = -1;
      for (int i : seq) {
        if (placed[i] || (prev[i] >= 0 && !placed[prev[i]])) continue;
        bool ready = true;
        for (int j : p.ops[i].waits[pass]) ready = ready && placed[j];
        if (!ready) continue;
        if (pick < 0 || level[i] > level[pick]) pick = i;
      }
      if (pick < 0) {  // cannot happen for a plan built above; keep pass order
        order = seq;
        break;
      }
      placed[pick] = 1;
      order.push_back(pick);
    }
  }
}

xpipe_status build_plan(const xpipe_layer_desc* L, int n, int mb, int H, int W, int C, int dtype,
                        Plan& p) {
  if (!L || n <= 0) return fail(XPIPE_EINVAL, "empty layer list");
  if (mb <= 0 || H <= 0 || W <= 0 || C <= 0) return fail(XPIPE_EINVAL, "bad input shape");
  if (dtype != DT_F32 && dtype != DT_BF16) return fail(XPIPE_EINVAL, "bad dtype");
  if ((int64_t)mb * H * W > (int64_t)1 << 30) return fail(XPIPE_EINVAL, "micro-batch too large");
  const size_t esz = dtype == DT_BF16 ? 2 : 4;

  // ---- shapes and parameters
  std::vector<Shape> sh(n);
  std::vector<int> consumers(n + 1, 0);  // index i+1 for layer i, 0 for the input
  Shape in{mb, H, W, C};
  auto shape_of = [&](int idx) -> Shape { return idx < 0 ? in : sh[idx]; };
  int64_t P = 0;
  std::vector<int64_t> poff(n, -1), poff2(n, -1);
  for (int i = 0; i < n; ++i) {
    const xpipe_layer_desc& d = L[i];
    char where[64];
    snprintf(where, sizeof where, "layer %d: ", i);
    int ni = d.n_inputs;
    int need = (d.kind == XPIPE_ADD) ? 2 : (d.kind == XPIPE_CONCAT ? -1 : 1);
    if (need > 0 && ni != need) return fail(XPIPE_EINVAL, std::string(where) + "wrong input count");
    if (d.kind == XPIPE_CONCAT && (ni < 2 || ni > XPIPE_MAX_INPUTS))
      return fail(XPIPE_EINVAL, std::string(where) + "concat takes 2..4 inputs");
    for (int j = 0; j < ni; ++j) {
      if (d.inputs[j] < -1 || d.inputs[j] >= i)
        return fail(XPIPE_EINVAL, std::string(where) + "input index out of order");
      consumers[d.inputs[j] + 1]++;
    }
    Shape s = shape_of(d.inputs[0]);
    switch (d.kind) {
      case XPIPE_LINEAR:
      case XPIPE_CONV: {
        const bool lin = d.kind == XPIPE_LINEAR;
        int k = lin ? 1 : d.k;
        int kw = lin ? 1 : (d.kw > 0 ? d.kw : d.k);
        if (lin && (s.H != 1 || s.W != 1))
          return fail(XPIPE_EINVAL, std::string(where) + "linear input must have H = W = 1");
        if (k < 1 || k > 7 || (k % 2) == 0 || kw < 1 || kw > 7 || (kw % 2) == 0)
          return fail(XPIPE_EINVAL, std::string(where) + "bad kernel size");
        if (d.stride < 0 || d.stride > 2 || (lin && d.stride > 1))
          return fail(XPIPE_EINVAL, std::string(where) + "stride must be 1 or 2 (convolutions only)");
        if (d.pad < 0 || d.pad > 1 || (lin && d.pad != 0))
          return fail(XPIPE_EINVAL, std::string(where) + "pad must be 0 (same) or 1 (none), convolutions only");
        if (d.cin != s.C || d.cout <= 0) return fail(XPIPE_EINVAL, std::string(where) + "channel mismatch");
        poff[i] = P;
        P += align_up((int64_t)d.cout * k * kw * d.cin, PARAM_ALIGN);
        if (d.has_bias) {
          poff2[i] = P;
          P += align_up(d.cout, PARAM_ALIGN);
        }
        s.C = d.cout;
        {
          const int st_ = d.stride == 2 ? 2 : 1;
          const int ph = d.pad ? 0 : k / 2, pw = d.pad ? 0 : kw / 2;
          const int Ho = (s.H + 2 * ph - k) / st_ + 1, Wo = (s.W + 2 * pw - kw) / st_ + 1;
          if (s.H + 2 * ph < k || s.W + 2 * pw < kw || Ho < 1 || Wo < 1)
            return fail(XPIPE_EINVAL, std::string(where) + "input smaller than the kernel");
          s.H = Ho;
          s.W = Wo;
        }
        break;
      }
      case XPIPE_BN:
        if (d.cout != s.C) return fail(XPIPE_EINVAL, std::string(where) + "bn channel mismatch");
        poff[i] = P;
        P += align_up(s.C, PARAM_ALIGN);
        poff2[i] = P;
        P += align_up(s.C, PARAM_ALIGN);
        break;
      case XPIPE_RELU:
        break;
      case XPIPE_ADD: {
        Shape s2 = shape_of(d.inputs[1]);
        if (s2.n != s.n || s2.H != s.H || s2.W != s.W || s2.C != s.C)
          return fail(XPIPE_EINVAL, std::string(where) + "add shape mismatch");
        break;
      }
      case XPIPE_MAXPOOL2:
        if (s.H < 2 || s.W < 2) return fail(XPIPE_EINVAL, std::string(where) + "maxpool input too small");
        s.H /= 2;
        s.W /= 2;
        break;
      case XPIPE_AVGPOOL3:
        break;
      case XPIPE_MAXPOOL3S2: {
        if (d.pad < 0 || d.pad > 1) return fail(XPIPE_EINVAL, std::string(where) + "bad pool padding");
        const int p_ = d.pad ? 0 : 1;
        if (s.H + 2 * p_ < 3 || s.W + 2 * p_ < 3)
          return fail(XPIPE_EINVAL, std::string(where) + "maxpool input too small");
        s.H = (s.H + 2 * p_ - 3) / 2 + 1;
        s.W = (s.W + 2 * p_ - 3) / 2 + 1;
        break;
      }
      case XPIPE_GAP:
        s.H = 1;
        s.W = 1;
        break;
      case XPIPE_CONCAT: {
        int c = 0;
        for (int j = 0; j < ni; ++j) {
          Shape sj = shape_of(d.inputs[j]);
          if (sj.n != s.n || sj.H != s.H || sj.W != s.W)
            return fail(XPIPE_EINVAL, std::string(where) + "concat spatial mismatch");
          c += sj.C;
        }
        s.C = c;
        break;
      }
      case XPIPE_SOFTMAX_CE:
        if (i != n - 1) return fail(XPIPE_EINVAL, std::string(where) + "softmax_ce must be last");
        if (s.H != 1 || s.W != 1 || d.classes != s.C || s.C <= 0)
          return fail(XPIPE_EINVAL, std::string(where) + "softmax_ce needs [n, classes] logits");
        if (s.n > 1024) return fail(XPIPE_EINVAL, std::string(where) + "micro-batch above 1024");
        break;
      default:
        return fail(XPIPE_EINVAL, std::string(where) + "unknown layer kind");
    }
    sh[i] = s;
  }
  for (int i = 0; i < n - 1; ++i)
    if (consumers[i + 1] == 0)
      return fail(XPIPE_EINVAL, "layer " + std::to_string(i) + " output is never used");
  if (consumers[0] == 0) return fail(XPIPE_EINVAL, "stage input is never used");

  // parameter table
  for (int i = 0; i < n; ++i) {
    const xpipe_layer_desc& d = L[i];
    if (d.kind == XPIPE_LINEAR || d.kind == XPIPE_CONV) {
      const int k = d.kind == XPIPE_LINEAR ? 1 : d.k;
      const int kw = d.kind == XPIPE_LINEAR ? 1 : (d.kw > 0 ? d.kw : d.k);
      p.params.push_back({poff[i], (int64_t)d.cout * k * kw * d.cin});
      if (d.has_bias) p.params.push_back({poff2[i], d.cout});
    } else if (d.kind == XPIPE_BN) {
      p.params.push_back({poff[i], d.cout});
      p.params.push_back({poff2[i], d.cout});
    }
  }
  p.P = P;

  // ---- grouping
  auto single_consumer = [&](int i, int kind) -> int {
    // index of the only consumer of layer i if it has the given kind, else -1
    if (consumers[i + 1] != 1) return -1;
    for (int j = i + 1; j < n; ++j)
      for (int q = 0; q < L[j].n_inputs; ++q)
        if (L[j].inputs[q] == i) return L[j].kind == kind ? j : -1;
    return -1;
  };
  std::vector<int> tensor_of(n, -1);  // layer -> tensor holding its (group's) output
  std::vector<bool> absorbed(n, false);
  p.tensors.clear();
  Tensor tin;
  tin.sh = in;
  p.tensors.push_back(tin);  // tensor 0: stage input
  auto tens = [&](int layer) -> int { return layer < 0 ? 0 : tensor_of[layer]; };
  auto new_tensor = [&](Shape s) -> int {
    Tensor t;
    t.sh = s;
    p.tensors.push_back(t);
    return (int)p.tensors.size() - 1;
  };

  for (int i = 0; i < n; ++i) {
    if (absorbed[i]) continue;
    const xpipe_layer_desc& d = L[i];
    Op op;
    op.layer = i;
    op.in = tens(d.inputs[0]);
    if (op.in < 0) return fail(XPIPE_EINVAL, "layer " + std::to_string(i) + " reads a fused intermediate");
    int last = i;
    switch (d.kind) {
      case XPIPE_LINEAR:
      case XPIPE_CONV: {
        op.kind = OP_GEMM;
        op.cin = d.cin;
        op.cout = d.cout;
        op.k = d.kind == XPIPE_LINEAR ? 1 : d.k;
        op.kw = d.kind == XPIPE_LINEAR ? 1 : (d.kw > 0 ? d.kw : d.k);
        op.stride = d.stride == 2 ? 2 : 1;
        op.ph = d.pad ? 0 : op.k / 2;
        op.pw = d.pad ? 0 : op.kw / 2;
        op.grid = op.stride > 1 || d.pad != 0;
        op.w_off = poff[i];
        op.b_off = d.has_bias ? poff2[i] : -1;
        int r = single_consumer(i, XPIPE_RELU);
        if (r >= 0) {
          op.relu = true;
          absorbed[r] = true;
          last = r;
        }
        break;
      }
      case XPIPE_BN: {
        op.kind = OP_BN;
        op.g_off = poff[i];
        op.be_off = poff2[i];
        int a = single_consumer(i, XPIPE_ADD);
        int other = a >= 0 ? (L[a].inputs[0] == i ? L[a].inputs[1] : L[a].inputs[0]) : -2;
        // the residual must already exist when the BN group runs
        if (a >= 0 && (other == i || other >= i)) a = -1;
        if (a >= 0) {
          op.in2 = tens(other);
          if (op.in2 < 0) return fail(XPIPE_EINVAL, "residual reads a fused intermediate");
          absorbed[a] = true;
          last = a;
        }
        int r = single_consumer(last, XPIPE_RELU);
        if (r >= 0) {
          op.relu = true;
          absorbed[r] = true;
          last = r;
        }
        break;
      }
      case XPIPE_ADD:
      case XPIPE_RELU: {
        op.kind = OP_ELT;
        if (d.kind == XPIPE_ADD) {
          op.in2 = tens(d.inputs[1]);
          if (op.in2 < 0) return fail(XPIPE_EINVAL, "add reads a fused intermediate");
        } else {
          op.relu = true;
        }
        if (d.kind == XPIPE_ADD) {
          int r = single_consumer(i, XPIPE_RELU);
          if (r >= 0) {
            op.relu = true;
            absorbed[r] = true;
            last = r;
          }
        }
        break;
      }
      case XPIPE_MAXPOOL2: op.kind = OP_MAXPOOL; break;
      case XPIPE_MAXPOOL3S2:
        op.kind = OP_MAXPOOL3;
        op.valid = d.pad != 0;
        break;
      case XPIPE_AVGPOOL3: op.kind = OP_AVGPOOL; break;
      case XPIPE_GAP: op.kind = OP_GAP; break;
      case XPIPE_CONCAT: op.kind = OP_CONCAT; break;
      case XPIPE_SOFTMAX_CE: op.kind = OP_CE; break;
    }
    if (op.kind != OP_CE) {
      int t = new_tensor(sh[last]);
      p.tensors[t].masked = op.relu;
      for (int q = i; q <= last; ++q)
        if (q == i || absorbed[q]) tensor_of[q] = t;
      op.out = t;
    }
    p.ops.push_back(op);
  }

  // consumer counts per tensor (by op inputs)
  for (const Op& op : p.ops) {
    if (op.kind == OP_CONCAT) {
      for (int q = 0; q < L[op.layer].n_inputs; ++q) p.tensors[tens(L[op.layer].inputs[q])].consumers++;
      continue;
    }
    p.tensors[op.in].consumers++;
    if (op.in2 >= 0) p.tensors[op.in2].consumers++;
  }

  // ---- concat views.  A max pool of ReLU outputs counts as masked: where its
  // output is 0 the whole window is 0, so masking its gradient there changes
  // nothing below the pool (the pooled ReLU outputs mask it anyway).
  for (const Op& op : p.ops) {
    if (op.kind == OP_MAXPOOL || op.kind == OP_MAXPOOL3) {
      p.tensors[op.out].masked = p.tensors[op.in].masked;
      continue;
    }
    if (op.kind != OP_CONCAT) continue;
    int coff = 0;
    bool all_masked = true, any_masked = false;
    for (int q = 0; q < L[op.layer].n_inputs; ++q) {
      int t = tens(L[op.layer].inputs[q]);
      Tensor& m = p.tensors[t];
      if (t == 0 || m.owner >= 0 || m.consumers != 1)
        return fail(XPIPE_EUNSUPPORTED, "concat inputs must be layer outputs used only by the concat");
      m.owner = op.out;
      m.coff = coff;
      coff += m.sh.C;
      all_masked = all_masked && m.masked;
      any_masked = any_masked || m.masked;
    }
    if (!all_masked && any_masked)
      return fail(XPIPE_EUNSUPPORTED,
                  "concat inputs must be all ReLU outputs or all not: the gradient of the concat "
                  "is masked as one tensor");
    p.tensors[op.out].masked = all_masked;
  }
  // concat-of-concat: resolve owners transitively
  for (size_t t = 0; t < p.tensors.size(); ++t) {
    int o = p.tensors[t].owner;
    while (o >= 0 && p.tensors[o].owner >= 0) {
      p.tensors[t].coff += p.tensors[o].coff;
      o = p.tensors[o].owner;
    }
    p.tensors[t].owner = o;
  }

  const Op& lastop = p.ops.back();
  if (lastop.kind == OP_CE) {
    p.has_loss = true;
    p.classes = L[n - 1].classes;
    p.out_tensor = lastop.in;
    if (p.tensors[p.out_tensor].consumers != 1 || p.tensors[p.out_tensor].masked ||
        p.tensors[p.out_tensor].owner >= 0 || p.out_tensor == 0)
      return fail(XPIPE_EUNSUPPORTED, "softmax_ce input must be a linear/conv output used only by it");
  } else {
    p.out_tensor = lastop.out;
  }

  // The merge below is exact in real arithmetic and leaves every forward
  // value bit for bit as the layer-by-layer launches give it, but the merged
  // data gradient adds the siblings' contributions before rounding once.  The
  // bf16 variant takes it; the fp32 variant keeps the rounding points of the
  // layer-by-layer definition.
  const bool rewrite = dtype == DT_BF16;

  // ---- sibling merge: convolutions with the same input and kernel size (no
  // bias, no fused ReLU, outputs not in a concat) become one GEMM launch whose
  // output is a buffer the siblings' outputs are channel slices of: the input
  // is read once, and the backward takes one data-gradient and one
  // weight-gradient launch for all of them
  for (size_t i = 0; rewrite && i < p.ops.size(); ++i) {
    auto mergeable = [&](const Op& o) {
      const Tensor& t = p.tensors[o.out];
      return o.kind == OP_GEMM && o.segs.empty() && o.b_off < 0 && !o.relu && t.owner < 0 &&
             o.out != p.out_tensor;
    };
    if (!mergeable(p.ops[i])) continue;
    std::vector<size_t> sib{i};
    for (size_t j = i + 1; j < p.ops.size() && sib.size() < (size_t)GATHER_MAX_SEGS; ++j)
      if (mergeable(p.ops[j]) && p.ops[j].in == p.ops[i].in && p.ops[j].k == p.ops[i].k &&
          p.ops[j].kw == p.ops[i].kw && p.ops[j].stride == p.ops[i].stride &&
          p.ops[j].grid == p.ops[i].grid)
        sib.push_back(j);
    if (sib.size() < 2) continue;
    Op m = p.ops[i];
    m.w_off = -1;
    m.cout = 0;
    for (size_t q : sib) m.cout += p.ops[q].cout;
    Shape ms = p.tensors[m.out].sh;
    ms.C = m.cout;
    const int owner = new_tensor(ms);
    p.tensors[owner].consumers = 1;
    int coff = 0;
    for (size_t q : sib) {
      const Op& o = p.ops[q];
      m.segs.push_back({o.w_off, o.cout});
      p.tensors[o.out].owner = owner;
      p.tensors[o.out].coff = coff;
      coff += o.cout;
    }
    m.out = owner;
    for (size_t k = sib.size() - 1; k >= 1; --k) p.ops.erase(p.ops.begin() + sib[k]);
    p.ops[i] = m;
  }

  // ---- batch-norm statistics fused into the producing conv / linear epilogue
  for (size_t i = 0; i < p.ops.size(); ++i) {
    Op& bn = p.ops[i];
    if (bn.kind != OP_BN || bn.in == 0) continue;
    const Tensor& z = p.tensors[bn.in];
    if (z.consumers != 1) continue;
    const int src = z.owner >= 0 ? z.owner : bn.in;
    for (size_t j = 0; j < i; ++j) {
      Op& g = p.ops[j];
      if (g.kind != OP_GEMM || g.out != src || g.relu) continue;
      // a view is only fed by a merged GEMM
      if (z.owner >= 0 && g.segs.empty()) continue;
      g.stats = true;
      bn.stats_fused = true;
      bn.stats_from = (int)j;
    }
  }

  // ---- the BNs over one merged GEMM's slices (statistics from its epilogue,
  // no residual) can be applied by one launch; taken when a pass runs as a
  // single chain of launches, where it removes launches without serialising
  // anything (with parallel lanes the separate launches let the branches start
  // apart, which measured faster)
  for (size_t j = 0; j < p.ops.size(); ++j) {
    const Op& g = p.ops[j];
    if (g.kind != OP_GEMM || g.segs.empty() || !g.stats) continue;
    std::vector<int> mem;
    bool ok = true;
    for (size_t i = 0; i < p.ops.size(); ++i) {
      const Op& bn = p.ops[i];
      if (bn.kind != OP_BN || !bn.stats_fused || bn.stats_from != (int)j || bn.in2 >= 0) continue;
      const Tensor& z = p.tensors[bn.in];
      ok = ok && z.coff % 8 == 0 && z.sh.C % 8 == 0;
      mem.push_back((int)i);
    }
    if (!ok || mem.size() < 2 || mem.size() > (size_t)BN_APPLY_SEGS) continue;
    for (int i : mem) p.ops[i].apply_grp = (int)p.apply_groups.size();
    p.apply_groups.push_back(mem);
  }

  // ---- backward accumulation order: walk ops in reverse; first contribution writes
  {
    std::vector<bool> written(p.tensors.size(), false);
    auto claim = [&](int t) -> bool {
      int o = p.tensors[t].owner >= 0 ? p.tensors[t].owner : t;
      // concat members are disjoint slices of their owner: track per member
      int key = p.tensors[t].owner >= 0 ? t : o;
      bool acc = written[key];
      written[key] = true;
      return acc;
    };
    for (int i = (int)p.ops.size() - 1; i >= 0; --i) {
      Op& op = p.ops[i];
      if (op.kind == OP_CONCAT) {
        // the gradient of the concat is, slice by slice, the gradient of its members
        for (int q = 0; q < L[op.layer].n_inputs; ++q) claim(tens(L[op.layer].inputs[q]));
        continue;
      }
      op.in_acc = claim(op.in);
      if (op.in2 >= 0) op.in2_acc = claim(op.in2);
    }
  }

  // ---- bf16: BN backward partials from the data-gradient epilogue of the GEMM
  // that completes the gradient of the BN outputs: a GEMM reading a whole
  // tensor (standalone or a concat) that is the first of the tensor's
  // readers, so the last writer of its gradient in the backward; the BNs
  // whose output is that tensor or a member of it take their partials from
  // the launch, at most CONV_BN_SEGS of them
  if (dtype == DT_BF16) {
    for (size_t j = 0; j < p.ops.size(); ++j) {
      Op& g = p.ops[j];
      const int t = g.in;
      // a GEMM's data gradient, or a global average pool's backward (the
      // classifier head's), can take the partials
      if ((g.kind != OP_GEMM && g.kind != OP_GAP) || t <= 0 || p.tensors[t].owner >= 0) continue;
      if (g.kind == OP_GAP && p.tensors[t].sh.C % 8 != 0) continue;
      const Region rt = region_of(p, t);
      bool first = true;
      for (size_t k = 0; k < j && first; ++k) {
        const Op& o = p.ops[k];
        if (o.kind == OP_CONCAT) continue;
        for (int r : {o.in, o.in2})
          if (r >= 0 && overlap(region_of(p, r), rt)) first = false;
      }
      if (!first) continue;
      std::vector<std::pair<int, int>> segs;
      for (size_t b = 0; b < p.ops.size(); ++b) {
        const Op& bn = p.ops[b];
        // BNs (with or without a residual: the partials are of the gradient
        // at the BN(+add) output either way), and, for a GEMM's epilogue,
        // convolutions with a bias (their bias gradient is the column sums of
        // the same g)
        const bool is_bn = bn.kind == OP_BN;
        const bool is_bias = g.kind == OP_GEMM && bn.kind == OP_GEMM && bn.b_off >= 0 && bn.segs.empty();
        if ((!is_bn && !is_bias) || bn.out == p.out_tensor) continue;
        const Tensor& u = p.tensors[bn.out];
        if (g.kind == OP_GAP && (u.coff % 8 != 0 || u.sh.C % 8 != 0)) continue;
        if (bn.out == t) segs.push_back({(int)b, 0});
        else if (u.owner == t) segs.push_back({(int)b, u.coff});
      }
      if (segs.empty() || segs.size() > (size_t)CONV_BN_SEGS) continue;
      g.bnb_segs = segs;
      for (auto& sg : segs) {
        p.ops[sg.first].bnb_gemm = (int)j;
        p.ops[sg.first].bnb_c0 = sg.second;
      }
    }
  }

  // ---- bf16: average pool -> 1x1 convolution, backward reordered (the
  // averaging runs on the convolution's cout channels instead of its cin)
  if (dtype == DT_BF16) {
    for (size_t a = 0; a < p.ops.size(); ++a) {
      Op& ap = p.ops[a];
      if (ap.kind != OP_AVGPOOL) continue;
      const int t = ap.out;
      if (t <= 0 || t == p.out_tensor || p.tensors[t].owner >= 0 || p.tensors[t].masked) continue;
      bool owns = false;
      for (const Tensor& u : p.tensors) owns = owns || u.owner == t;
      if (owns) continue;
      int user = -1, users = 0;
      for (size_t j = 0; j < p.ops.size(); ++j) {
        const Op& o = p.ops[j];
        if (o.kind == OP_CONCAT) continue;
        if (o.in == t || o.in2 == t) {
          ++users;
          user = (int)j;
        }
      }
      if (users != 1) continue;
      Op& g = p.ops[user];
      if (g.kind != OP_GEMM || g.in != t || g.in2 >= 0 || g.k != 1 || g.kw != 1 || g.grid ||
          !g.segs.empty() || !g.bnb_segs.empty())
        continue;
      g.pool_bwd = (int)a;
      ap.pool_by = user;
    }
  }

  // ---- launch lanes
  plan_lanes(p);
  if (const char* tr = std::getenv("XPIPE_TRACE_PLAN"); tr && *tr == '1') {
    static const char* kn[] = {"gemm", "bn", "elt", "maxpool", "avgpool", "gap", "concat", "ce", "maxpool3"};
    for (size_t i = 0; i < p.ops.size(); ++i) {
      const Op& o = p.ops[i];
      std::fprintf(stderr, "op %2zu %-7s layer %2d in %2d out %2d cout %3d segs %zu | fwd lane %d waits",
                   i, kn[o.kind], o.layer, o.in, o.out, o.cout, o.segs.size(), o.lane[0]);
      for (int j : o.waits[0]) std::fprintf(stderr, " %d", j);
      std::fprintf(stderr, " | bwd lane %d waits", o.lane[1]);
      for (int j : o.waits[1]) std::fprintf(stderr, " %d", j);
      std::fprintf(stderr, "\n");
    }
  }

  // ---- workspace layout
  size_t off = 0;
  auto take = [&](size_t bytes) -> int64_t {
    off = (size_t)align_up((int64_t)off, WS_ALIGN);
    int64_t at = (int64_t)off;
    off += bytes;
    return at;
  };
  if (dtype == DT_BF16) {
    p.bf_f_off = take((size_t)P * 2);
    p.bf_b_off = take((size_t)P * 2);
  }
  size_t colpart = 0, wpart = 0;
  for (Op& op : p.ops) {
    const Tensor& tin_ = p.tensors[op.in];
    if (op.kind == OP_GEMM) {
      op.wd_off = take((size_t)op.cout * op.k * op.kw * op.cin * esz);
      if (!op.segs.empty())
        for (int d = 0; d < 2; ++d)
          op.wg_off[d] = take((size_t)op.cout * op.k * op.kw * op.cin * esz);
      if (op.stats) op.stat_block = take((size_t)4 * op.cout * sizeof(double));
      if (op.pool_bwd >= 0)
        op.box_off = take((size_t)p.tensors[op.out].sh.rows() * op.cout * esz);
      if (!op.bnb_segs.empty())
        op.bnb_part_off = take((size_t)conv_max_row_tiles((int)tin_.sh.rows()) * 2 * op.cin * sizeof(double));
      int M = (int)p.tensors[op.out].sh.rows();  // output pixels (the input's for stride 1)
      int K = op.k * op.kw * op.cin;
      int splits = wgrad_pick_splits(dtype, M, op.cout, K, op.k * op.kw);
      wpart = std::max(wpart, wgrad_part_bytes(dtype, op.cout, K, splits));
      if (op.b_off >= 0) colpart = std::max(colpart, col_partial_bytes(M, op.cout));
      if (op.stats)
        colpart = std::max(colpart, (size_t)conv_max_row_tiles(M) * 2 * op.cout * sizeof(double));
    } else if (op.kind == OP_BN) {
      if (op.stats_fused) {
        // the GEMM's statistics block, at this BN's channels
        const Op& g = p.ops[op.stats_from];
        op.stat_off = g.stat_block + (int64_t)tin_.coff * (int64_t)sizeof(double);
        op.stat_ld = g.cout;
      } else {
        op.stat_off = take((size_t)4 * tin_.sh.C * sizeof(double));
        op.stat_ld = tin_.sh.C;
      }
      colpart = std::max(colpart, col_partial_bytes((int)tin_.sh.rows(), tin_.sh.C));
    } else if (op.kind == OP_GAP) {
      colpart = std::max(colpart, gap_partial_bytes(tin_.sh.n, tin_.sh.H, tin_.sh.W, tin_.sh.C));
      if (!op.bnb_segs.empty())
        op.bnb_part_off = take((size_t)gap_bn_max_row_blocks() * 2 * tin_.sh.C * sizeof(double));
    } else if (op.kind == OP_MAXPOOL3) {
      op.idx_off = take((size_t)p.tensors[op.out].sh.elems());
    }
  }
  for (size_t t = 1; t < p.tensors.size(); ++t) {
    Tensor& tt = p.tensors[t];
    if (tt.owner >= 0) continue;
    tt.act_off = take((size_t)tt.sh.elems() * esz);
    tt.grad_off = take((size_t)tt.sh.elems() * esz);
  }
  for (int l = 0; l < NLANES; ++l) {
    p.colpart_off[l] = take(std::max<size_t>(colpart, 64));
    p.wpart_off[l] = take(std::max<size_t>(wpart, 64));
  }
  p.ws = (size_t)align_up((int64_t)off, WS_ALIGN);
  return XPIPE_OK;
}

// ============================================================================
// execution helpers
// ============================================================================
struct View {
  char* p;
  int ld;
};

struct Ctx {
  const void* x = nullptr;  // stage input
  void* y = nullptr;        // stage output override (forward)
  void* dx = nullptr;       // stage input gradient (backward), may be null
};

View act(xpipe_stage* st, int t, const Ctx& c) {
  const Tensor& tt = st->tensors[t];
  if (t == 0) return View{(char*)c.x, tt.sh.C};
  int o = tt.owner >= 0 ? tt.owner : t;
  const Tensor& ot = st->tensors[o];
  char* base = (c.y && o == st->out_tensor) ? (char*)c.y : st->ws + ot.act_off;
  return View{base + (size_t)tt.coff * st->esz(), ot.sh.C};
}

View gradv(xpipe_stage* st, int t, const Ctx& c) {
  const Tensor& tt = st->tensors[t];
  if (t == 0) return View{(char*)c.dx, tt.sh.C};
  int o = tt.owner >= 0 ? tt.owner : t;
  const Tensor& ot = st->tensors[o];
  return View{st->ws + ot.grad_off + (size_t)tt.coff * st->esz(), ot.sh.C};
}

hipEvent_t take_event(xpipe_stage* st) {
  if (!st->pool.empty()) {
    hipEvent_t e = st->pool.back();
    st->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

void xpipe_stage::Hook::before() {
  a = take_event(st);
  if (a) (void)hipEventRecord(a, st->stream);
}

void xpipe_stage::Hook::after(const char* name, double work) {
  if (!a) return;
  hipEvent_t b = take_event(st);
  if (!b) {
    st->pool.push_back(a);
    a = nullptr;
    return;
  }
  (void)hipEventRecord(b, st->stream);
  st->pending.push_back(TimeRec{a, b, name, work});
  a = nullptr;
}

namespace {

// installs the stage's launch observer for the duration of one ABI call
struct HookScope {
  HookScope(xpipe_stage* st) { xp::g_hook = st->timing ? &st->hook : nullptr; }
  ~HookScope() { xp::g_hook = nullptr; }
};

const void* gemm_weights(xpipe_stage* st, const Op& op, int dir) {
  if (!op.segs.empty()) return st->wws + op.wg_off[dir];
  if (st->dtype == DT_BF16) {
    int64_t off = dir == XPIPE_FWD ? st->bf_f_off : st->bf_b_off;
    return st->wws + off + (size_t)op.w_off * 2;
  }
  return (dir == XPIPE_FWD ? st->wpf : st->wpb) + op.w_off;
}

const float* fp32_param(xpipe_stage* st, int64_t off, int dir) {
  return (dir == XPIPE_FWD ? st->wpf : st->wpb) + off;
}


// ---------------------------------------------------------------- lanes
// One pass (forward or backward) over the ops, spread over the launch lanes.
#define XP_OK(call)                        \
  do {                                     \
    xpipe_status s_ = (call);              \
    if (s_ != XPIPE_OK) return s_;         \
  } while (0)

// With per-launch timing on, everything runs on the stage's stream.  While a
// pass is being recorded, every launch goes to the capture stream and the
// lanes become graph edges instead of events: before an op's first launch the
// capture's dependency set is replaced by the last nodes of the op's lane and
// of the ops it waits for, so the recorded graph has the same ordering as the
// multi-stream execution (per-lane scratch still follows the op's lane).
struct Lanes {
  typedef std::vector<hipGraphNode_t> Nodes;
  xpipe_stage* st;
  int pass;
  bool used[NLANES] = {};
  bool forked = false;
  Nodes ltail[NLANES];        // recording: last nodes per lane
  std::vector<Nodes> otail;  // recording: last nodes of each op
  bool started = false;
  bool chain = false;  // every op on lane 0, in order
  Lanes(xpipe_stage* st_, int pass_, bool chain_ = false) : st(st_), pass(pass_), chain(chain_) {}
  // recording: every lane starts after everything captured so far (the
  // graph itself starts after the work enqueued before its launch)
  xpipe_status start() {
    if (started) return XPIPE_OK;
    started = true;
    otail.resize(st->ops.size());
    XP_OK(capture_tail(ltail[0]));
    for (int l = 1; l < NLANES; ++l) ltail[l] = ltail[0];
    return XPIPE_OK;
  }
  xpipe_status capture_tail(Nodes& out) {
    hipStreamCaptureStatus cs;
    const hipGraphNode_t* d = nullptr;
    size_t nd = 0;
    XP_HIP(hipStreamGetCaptureInfo_v2(st->cap_stream, &cs, nullptr, nullptr, &d, &nd));
    out.assign(d, d + nd);
    return XPIPE_OK;
  }
  bool single() const { return st->timing || st->one_lane || chain; }
  // stream for op i after its waits; the first use of an auxiliary lane in
  // the pass waits for the work enqueued on the stage's stream before it
  xpipe_status begin(int i, hipStream_t& s, int& lane) {
    const Op& op = st->ops[i];
    lane = single() ? 0 : op.lane[pass];
    if (st->capturing) {
      XP_OK(start());
      s = st->cap_stream;
      used[lane] = true;
      Nodes d = ltail[lane];
      if (!single())
        for (int j : op.waits[pass])
          for (hipGraphNode_t n : otail[j])
            if (std::find(d.begin(), d.end(), n) == d.end()) d.push_back(n);
      XP_HIP(hipStreamUpdateCaptureDependencies(s, d.data(), d.size(), hipStreamSetCaptureDependencies));
      return XPIPE_OK;
    }
    s = st->lane_stream[lane];
    if (lane > 0 && !used[lane]) {
      if (!forked) XP_HIP(hipEventRecord(st->fork_ev, st->stream));
      forked = true;
      XP_HIP(hipStreamWaitEvent(s, st->fork_ev, 0));
    }
    used[lane] = true;
    if (!single())
      for (int j : op.waits[pass]) XP_HIP(hipStreamWaitEvent(s, st->op_ev[pass][j], 0));
    return XPIPE_OK;
  }
  // op i has completed what the ops waiting for it read (a backward GEMM's
  // input gradient): they wait for this point, not for the op's end
  std::vector<char> marked;
  xpipe_status mark(int i, hipStream_t s) {
    if (marked.empty()) marked.assign(st->ops.size(), 0);
    marked[i] = 1;
    if (st->capturing) return capture_tail(otail[i]);
    if (!single() && st->ops[i].record[pass]) XP_HIP(hipEventRecord(st->op_ev[pass][i], s));
    return XPIPE_OK;
  }
  xpipe_status end(int i, hipStream_t s) {
    const bool mk = !marked.empty() && marked[i];
    if (st->capturing) {
      (void)s;
      Nodes t;
      XP_OK(capture_tail(t));
      if (!mk) otail[i] = t;
      ltail[single() ? 0 : st->ops[i].lane[pass]] = t;
      return XPIPE_OK;
    }
    if (!mk && !single() && st->ops[i].record[pass]) XP_HIP(hipEventRecord(st->op_ev[pass][i], s));
    return XPIPE_OK;
  }
  // the stage's stream waits for every auxiliary lane used in the pass
  xpipe_status join() {
    if (st->capturing) {
      if (!started) return XPIPE_OK;
      Nodes all;
      for (int l = 0; l < NLANES; ++l)
        if (used[l] || l == 0)
          for (hipGraphNode_t n : ltail[l])
            if (std::find(all.begin(), all.end(), n) == all.end()) all.push_back(n);
      XP_HIP(hipStreamUpdateCaptureDependencies(st->cap_stream, all.data(), all.size(),
                                                hipStreamSetCaptureDependencies));
      return XPIPE_OK;
    }
    for (int l = 1; l < NLANES; ++l)
      if (used[l]) {
        XP_HIP(hipEventRecord(st->join_ev[l], st->lane_stream[l]));
        XP_HIP(hipStreamWaitEvent(st->stream, st->join_ev[l], 0));
      }
    return XPIPE_OK;
  }
};

// op order of a pass: pass order, or the interleaved order while recording
std::vector<int> pass_order(const xpipe_stage* st, int pass) {
  if (st->capturing) return st->rec_order[pass];
  const int n = (int)st->ops.size();
  std::vector<int> o(n);
  for (int q = 0; q < n; ++q) o[q] = pass == 0 ? q : n - 1 - q;
  return o;
}

// ---------------------------------------------------------------- forward
xpipe_status run_forward(xpipe_stage* st, int dir, const Ctx& c, const int32_t* labels,
                         float* loss, bool chain = false) {
  const int dt = st->dtype;
  Lanes lanes(st, 0, chain);
  // as one chain, a group of BNs is applied by one launch at its first member
  std::vector<char> grp_done(chain ? st->apply_groups.size() : 0, 0);
  for (int i : pass_order(st, 0)) {
    const Op& op = st->ops[i];
    if (op.kind == OP_CONCAT) continue;
    hipStream_t s;
    int lane;
    XP_OK(lanes.begin(i, s, lane));
    const Tensor& tin = st->tensors[op.in];
    View x = act(st, op.in, c);
    switch (op.kind) {
      case OP_GEMM: {
        View y = act(st, op.out, c);
        ConvArgs a{};
        a.x = x.p;
        a.ldx = x.ld;
        a.w = gemm_weights(st, op, dir);
        a.y = y.p;
        a.ldy = y.ld;
        a.bias = op.b_off >= 0 ? fp32_param(st, op.b_off, dir) : nullptr;
        a.nb = tin.sh.n;
        a.H = tin.sh.H;
        a.W = tin.sh.W;
        a.C = op.cin;
        a.N = op.cout;
        a.R = op.k;
        a.S = op.kw;
        a.pad = op.ph;
        a.padw = op.pw;
        a.relu = op.relu;
        const Tensor& tout = st->tensors[op.out];
        a.stride = op.stride;
        if (op.grid) {
          a.Ho = tout.sh.H;
          a.Wo = tout.sh.W;
        }
        int rows_tiles = 0;
        if (op.stats) a.stat_part = (double*)(st->ws + st->colpart_off[lane]);
        XP_HIP(launch_conv_gemm(dt, a, s, &rows_tiles));
        if (op.stats) {
          // the following BNs' batch statistics from the epilogue's column sums
          double* stats = (double*)(st->ws + op.stat_block);
          ColArgs ca{};
          ca.mode = COL_STATS;
          ca.M = (int)tout.sh.rows();
          ca.C = op.cout;
          ca.partial = a.stat_part;
          ca.row_blocks = rows_tiles;
          ca.out0 = stats;
          ca.out1 = stats + op.cout;
          ca.eps = BN_EPS;
          XP_HIP(launch_colfinal(ca, s));
        }
        break;
      }
      case OP_BN: {
        if (chain && op.apply_grp >= 0) {
          if (grp_done[op.apply_grp]) break;
          grp_done[op.apply_grp] = 1;
          const std::vector<int>& mem = st->apply_groups[op.apply_grp];
          const Op& g = st->ops[op.stats_from];
          const double* gst = (const double*)(st->ws + g.stat_block);
          View z = act(st, g.out, c);
          BnApplyArgs b{};
          b.z = z.p;
          b.ldz = z.ld;
          b.mean = gst;
          b.rstd = gst + g.cout;
          b.M = (int)tin.sh.rows();
          b.C = g.cout;
          b.nseg = (int)mem.size();
          for (int q = 0; q < b.nseg; ++q) {
            const Op& bn = st->ops[mem[q]];
            const Tensor& zt = st->tensors[bn.in];
            View y = act(st, bn.out, c);
            b.seg_c0[q] = zt.coff;
            b.seg_c1[q] = zt.coff + zt.sh.C;
            b.seg_y[q] = y.p;
            b.seg_ldy[q] = y.ld;
            b.seg_gamma[q] = fp32_param(st, bn.g_off, dir);
            b.seg_beta[q] = fp32_param(st, bn.be_off, dir);
            b.seg_relu[q] = bn.relu;
          }
          XP_HIP(launch_bn_apply(dt, b, s));
          break;
        }
        double* stats = (double*)(st->ws + op.stat_off);
        ColArgs ca{};
        ca.mode = COL_STATS;
        ca.a = x.p;
        ca.lda = x.ld;
        ca.M = (int)tin.sh.rows();
        ca.C = tin.sh.C;
        ca.partial = (double*)(st->ws + st->colpart_off[lane]);
        ca.row_blocks = col_row_blocks(ca.M, ca.C);
        ca.out0 = stats;
        ca.out1 = stats + op.stat_ld;
        ca.eps = BN_EPS;
        if (!op.stats_fused) {
          XP_HIP(launch_colreduce(dt, ca, s));
        }
        View y = act(st, op.out, c);
        BnApplyArgs b{};
        b.z = x.p;
        b.ldz = x.ld;
        b.mean = stats;
        b.rstd = stats + op.stat_ld;
        b.gamma = fp32_param(st, op.g_off, dir);
        b.beta = fp32_param(st, op.be_off, dir);
        if (op.in2 >= 0) {
          View r = act(st, op.in2, c);
          b.res = r.p;
          b.ldres = r.ld;
        }
        b.y = y.p;
        b.ldy = y.ld;
        b.M = ca.M;
        b.C = ca.C;
        b.relu = op.relu;
        XP_HIP(launch_bn_apply(dt, b, s));
        break;
      }
      case OP_ELT: {
        View y = act(st, op.out, c);
        EltArgs e{};
        e.a = x.p;
        e.lda = x.ld;
        if (op.in2 >= 0) {
          View b = act(st, op.in2, c);
          e.b = b.p;
          e.ldb = b.ld;
        }
        e.y = y.p;
        e.ldy = y.ld;
        e.M = (int)tin.sh.rows();
        e.C = tin.sh.C;
        e.relu = op.relu;
        XP_HIP(launch_elementwise(dt, e, s));
        break;
      }
      case OP_MAXPOOL:
      case OP_MAXPOOL3:
      case OP_AVGPOOL:
      case OP_GAP: {
        View y = act(st, op.out, c);
        PoolArgs pa{};
        pa.x = x.p;
        pa.ldx = x.ld;
        pa.out = y.p;
        pa.ldo = y.ld;
        pa.nb = tin.sh.n;
        pa.H = tin.sh.H;
        pa.W = tin.sh.W;
        pa.C = tin.sh.C;
        pa.valid = op.valid;
        pa.part = (double*)(st->ws + st->colpart_off[lane]);
        if (op.kind == OP_MAXPOOL3 && dir == XPIPE_BWD) {
          // the backward that follows this recomputation takes the choices
          pa.idx = (uint8_t*)(st->ws + op.idx_off);
          pa.ldi = tin.sh.C;
        }
        if (op.kind == OP_MAXPOOL) XP_HIP(launch_maxpool_fwd(dt, pa, s));
        else if (op.kind == OP_MAXPOOL3) XP_HIP(launch_maxpool3s2_fwd(dt, pa, s));
        else if (op.kind == OP_AVGPOOL) XP_HIP(launch_avgpool_fwd(dt, pa, s));
        else XP_HIP(launch_gap_fwd(dt, pa, s));
        break;
      }
      case OP_CONCAT:
        break;
      case OP_CE: {
        if (!loss) break;  // the forward of a loss stage needs no more than the logits
        CeArgs ce{};
        ce.z = x.p;
        ce.ldz = x.ld;
        ce.labels = labels;
        ce.n = tin.sh.n;
        ce.classes = st->classes;
        ce.inv_N = 1.0 / ((double)st->T * st->mb);
        ce.loss = loss;
        XP_HIP(launch_softmax_ce(dt, ce, s));
        break;
      }
    }
    XP_OK(lanes.end(i, s));
  }
  return lanes.join();
}

// ---------------------------------------------------------------- backward
xpipe_status run_backward(xpipe_stage* st, const Ctx& c, const void* dy, const int32_t* labels) {
  hipStream_t s = st->stream;
  int lane = 0;
  const int dt = st->dtype;
  const int dir = XPIPE_BWD;
  const size_t esz = st->esz();
  auto want_grad = [&](int t) { return t != 0 || c.dx != nullptr; };
  auto mask_of = [&](int t, const void*& mp, int& ld) {
    mp = nullptr;
    ld = 0;
    if (st->tensors[t].masked) {
      View v = act(st, t, c);
      mp = v.p;
      ld = v.ld;
    }
  };

  // seed: the gradient of the stage output
  if (!st->has_loss) {
    const Tensor& to = st->tensors[st->out_tensor];
    View g = gradv(st, st->out_tensor, c);
    EltArgs e{};
    e.a = dy;
    e.lda = to.sh.C;
    mask_of(st->out_tensor, e.mask, e.ldm);
    e.y = g.p;
    e.ldy = g.ld;
    e.M = (int)to.sh.rows();
    e.C = to.sh.C;
    XP_HIP(launch_elementwise(dt, e, s));
  }

  Lanes lanes(st, 1);
  for (int i : pass_order(st, 1)) {
    const Op& op = st->ops[i];
    if (op.kind == OP_CONCAT) continue;
    XP_OK(lanes.begin(i, s, lane));
    const Tensor& tin = st->tensors[op.in];
    View x = act(st, op.in, c);
    switch (op.kind) {
      case OP_CE: {
        View g = gradv(st, op.in, c);
        CeArgs ce{};
        ce.z = x.p;
        ce.ldz = x.ld;
        ce.labels = labels;
        ce.n = tin.sh.n;
        ce.classes = st->classes;
        ce.inv_N = 1.0 / ((double)st->T * st->mb);
        ce.dz = g.p;
        ce.lddz = g.ld;
        XP_HIP(launch_softmax_ce(dt, ce, s));
        break;
      }
      case OP_GEMM: {
        View g = gradv(st, op.out, c);
        const Tensor& tout = st->tensors[op.out];
        const int M = (int)tout.sh.rows();  // output pixels
        const int K = op.k * op.kw * op.cin;
        const Op* pool = op.pool_bwd >= 0 ? &st->ops[op.pool_bwd] : nullptr;
        if (pool ? want_grad(pool->in) : want_grad(op.in)) {
          View dx = gradv(st, pool ? pool->in : op.in, c);
          ConvArgs a{};
          a.x = g.p;
          a.ldx = g.ld;
          a.w = st->wws + op.wd_off;
          a.y = dx.p;
          a.ldy = dx.ld;
          mask_of(pool ? pool->in : op.in, a.mask, a.ldm);
          if (pool) {
            // the average pool's backward: average the output gradient over
            // 3x3 windows (cout channels), then the 1x1 data gradient writes
            // the pool input's gradient with the pool's mask and accumulation
            PoolArgs pa{};
            pa.x = g.p;
            pa.ldx = g.ld;
            pa.out = st->ws + op.box_off;
            pa.ldo = op.cout;
            pa.nb = tout.sh.n;
            pa.H = tout.sh.H;
            pa.W = tout.sh.W;
            pa.C = op.cout;
            XP_HIP(launch_avgpool_fwd(dt, pa, s));
            a.x = st->ws + op.box_off;
            a.ldx = op.cout;
          }
          a.nb = tin.sh.n;
          a.H = tin.sh.H;
          a.W = tin.sh.W;
          a.C = op.cout;
          a.N = op.cin;
          a.R = op.k;
          a.S = op.kw;
          a.pad = op.ph;
          a.padw = op.pw;
          a.accumulate = pool ? pool->in_acc : op.in_acc;
          if (op.grid) {
            // rows: the input grid; gathered from the output gradient's grid,
            // with the transposed (unflipped) weights
            a.tr = 1;
            a.stride = op.stride;
            a.H = tout.sh.H;
            a.W = tout.sh.W;
            a.Ho = tin.sh.H;
            a.Wo = tin.sh.W;
          }
          if (!op.bnb_segs.empty()) {
            // the batch norms whose output gradient this launch completes
            a.bn_part = (double*)(st->ws + op.bnb_part_off);
            a.bn_nseg = (int)op.bnb_segs.size();
            for (int k = 0; k < a.bn_nseg; ++k) {
              const Op& bn = st->ops[op.bnb_segs[k].first];
              a.bn_c0[k] = op.bnb_segs[k].second;
              if (bn.kind == OP_GEMM) {  // a convolution's bias: sums of g only
                a.bn_c1[k] = a.bn_c0[k] + bn.cout;
                a.bn_z[k] = nullptr;
                continue;
              }
              View z = act(st, bn.in, c);
              const double* bst = (const double*)(st->ws + bn.stat_off);
              a.bn_c1[k] = a.bn_c0[k] + st->tensors[bn.in].sh.C;
              a.bn_z[k] = z.p;
              a.ld_bnz[k] = z.ld;
              a.bn_mean[k] = bst;
              a.bn_rstd[k] = bst + bn.stat_ld;
            }
          }
          int rows_tiles = 0;
          XP_HIP(launch_conv_gemm(dt, a, s, &rows_tiles));
          if (!op.bnb_segs.empty()) st->bnb_nrb[i] = rows_tiles;
        }
        // the ops that wait for this one need only the input gradient (the
        // weight gradient is joined at the end of the pass): they are released
        // here, and the weight gradient follows on this lane (0.08 ms per
        // Inception-A step)
        XP_OK(lanes.mark(i, s));
        // weight gradient, accumulated into grad
        WgradArgs w{};
        w.dz = g.p;
        w.lddz = g.ld;
        w.x = x.p;
        w.ldx = x.ld;
        w.part = st->ws + st->wpart_off[lane];
        if (op.segs.empty()) {
          w.grad = st->grad + op.w_off;
        } else {
          w.nseg = (int)op.segs.size();
          int r0 = 0;
          for (int q = 0; q < w.nseg; ++q) {
            w.seg_row0[q] = r0;
            w.seg_grad[q] = st->grad + op.segs[q].first;
            r0 += op.segs[q].second;
          }
          w.seg_row0[w.nseg] = r0;
        }
        w.nb = tin.sh.n;
        w.H = tin.sh.H;
        w.W = tin.sh.W;
        w.C = op.cin;
        w.N = op.cout;
        w.R = op.k;
        w.S = op.kw;
        w.pad = op.ph;
        w.padw = op.pw;
        w.stride = op.stride;
        if (op.grid) {
          w.Ho = tout.sh.H;
          w.Wo = tout.sh.W;
        }
        w.splits = wgrad_pick_splits(dt, M, op.cout, K, op.k * op.kw);
        {
          XP_HIP(launch_wgrad(dt, w, s));
        }
        if (op.b_off >= 0) {
          ColArgs ca{};
          ca.mode = COL_BIAS;
          ca.a = g.p;
          ca.lda = g.ld;
          ca.M = M;
          ca.C = op.cout;
          ca.grad0 = st->grad + op.b_off;
          if (op.bnb_gemm >= 0) {
            // the column sums of g from the epilogue that completed it
            ca.row_blocks = st->bnb_nrb[op.bnb_gemm];
            ca.partial = (double*)(st->ws + st->ops[op.bnb_gemm].bnb_part_off) +
                         (size_t)op.bnb_c0 * 2 * ca.row_blocks;
            XP_HIP(launch_colfinal(ca, s));
          } else {
            ca.partial = (double*)(st->ws + st->colpart_off[lane]);
            ca.row_blocks = col_row_blocks(M, op.cout);
            XP_HIP(launch_colreduce(dt, ca, s));
          }
        }
        break;
      }
      case OP_BN: {
        View g = gradv(st, op.out, c);
        double* stats = (double*)(st->ws + op.stat_off);
        const int M = (int)tin.sh.rows(), C = tin.sh.C;
        ColArgs ca{};
        ca.mode = COL_BNBWD;
        ca.a = g.p;
        ca.lda = g.ld;
        ca.z = x.p;
        ca.ldz = x.ld;
        const int ld = op.stat_ld;
        ca.mean = stats;
        ca.rstd = stats + ld;
        ca.M = M;
        ca.C = C;
        ca.partial = (double*)(st->ws + st->colpart_off[lane]);
        ca.row_blocks = col_row_blocks(M, C);
        ca.out0 = stats + 2 * ld;
        ca.out1 = stats + 3 * ld;
        ca.grad0 = st->grad + op.g_off;
        ca.grad1 = st->grad + op.be_off;
        if (op.bnb_gemm >= 0) {
          // partials from the data-gradient epilogue that wrote g
          ca.row_blocks = st->bnb_nrb[op.bnb_gemm];
          ca.partial = (double*)(st->ws + st->ops[op.bnb_gemm].bnb_part_off) +
                       (size_t)op.bnb_c0 * 2 * ca.row_blocks;
          XP_HIP(launch_colfinal(ca, s));
        } else {
          XP_HIP(launch_colreduce(dt, ca, s));
        }
        BnBwdArgs b{};
        b.g = g.p;
        b.ldg = g.ld;
        b.z = x.p;
        b.ldz = x.ld;
        b.mean = stats;
        b.rstd = stats + ld;
        b.dbeta = stats + 2 * ld;
        b.dgamma = stats + 3 * ld;
        b.gamma = fp32_param(st, op.g_off, dir);
        bool need_dz = want_grad(op.in);
        View dz = gradv(st, op.in, c);
        b.dz = need_dz ? dz.p : nullptr;
        b.lddz = dz.ld;
        mask_of(op.in, b.dzmask, b.ldzm);
        b.dz_accumulate = op.in_acc;
        if (op.in2 >= 0 && want_grad(op.in2)) {
          View dr = gradv(st, op.in2, c);
          b.dres = dr.p;
          b.lddres = dr.ld;
          mask_of(op.in2, b.resmask, b.ldrm);
          b.res_accumulate = op.in2_acc;
        }
        b.M = M;
        b.C = C;
        if (!need_dz) {
          // no BN-input gradient wanted (stage input without dx): only the
          // residual part, as a masked copy
          if (b.dres) {
            EltArgs e{};
            e.a = g.p;
            e.lda = g.ld;
            e.mask = b.resmask;
            e.ldm = b.ldrm;
            e.y = b.dres;
            e.ldy = b.lddres;
            e.M = M;
            e.C = C;
            e.accumulate = b.res_accumulate;
            XP_HIP(launch_elementwise(dt, e, s));
          }
          break;
        }
        XP_HIP(launch_bn_bwd(dt, b, s));
        break;
      }
      case OP_ELT: {
        View g = gradv(st, op.out, c);
        int ins[2] = {op.in, op.in2};
        bool accs[2] = {op.in_acc, op.in2_acc};
        for (int q = 0; q < 2; ++q) {
          if (ins[q] < 0 || !want_grad(ins[q])) continue;
          View d = gradv(st, ins[q], c);
          EltArgs e{};
          e.a = g.p;
          e.lda = g.ld;
          mask_of(ins[q], e.mask, e.ldm);
          e.y = d.p;
          e.ldy = d.ld;
          e.M = (int)tin.sh.rows();
          e.C = tin.sh.C;
          e.accumulate = accs[q];
          XP_HIP(launch_elementwise(dt, e, s));
        }
        break;
      }
      case OP_MAXPOOL:
      case OP_MAXPOOL3:
      case OP_AVGPOOL:
      case OP_GAP: {
        if (!want_grad(op.in) || op.pool_by >= 0) break;  // (or taken by its 1x1 convolution)
        View g = gradv(st, op.out, c);
        View d = gradv(st, op.in, c);
        PoolArgs pa{};
        pa.x = x.p;
        pa.ldx = x.ld;
        pa.dy = g.p;
        pa.lddy = g.ld;
        pa.out = d.p;
        pa.ldo = d.ld;
        mask_of(op.in, pa.mask, pa.ldm);
        pa.accumulate = op.in_acc;
        pa.nb = tin.sh.n;
        pa.H = tin.sh.H;
        pa.W = tin.sh.W;
        pa.C = tin.sh.C;
        pa.valid = op.valid;
        if (op.kind == OP_MAXPOOL3) {
          // a pixel takes a window's gradient when it holds the window's
          // maximum first: the recomputed forward recorded that position
          pa.idx = (uint8_t*)(st->ws + op.idx_off);
          pa.ldi = tin.sh.C;
        }
        if (op.kind == OP_MAXPOOL) XP_HIP(launch_maxpool_bwd(dt, pa, s));
        else if (op.kind == OP_MAXPOOL3) XP_HIP(launch_maxpool3s2_bwd(dt, pa, s));
        else if (op.kind == OP_AVGPOOL) XP_HIP(launch_avgpool_bwd(dt, pa, s));
        else if (op.bnb_segs.empty()) XP_HIP(launch_gap_bwd(dt, pa, s));
        else {
          // with the backward partials of the batch norms whose output
          // gradient this completes
          GapBnArgs gb{};
          gb.part = (double*)(st->ws + op.bnb_part_off);
          gb.bn_nseg = (int)op.bnb_segs.size();
          for (int k = 0; k < gb.bn_nseg; ++k) {
            const Op& bn = st->ops[op.bnb_segs[k].first];
            View z = act(st, bn.in, c);
            const double* bst = (const double*)(st->ws + bn.stat_off);
            gb.bn_c0[k] = op.bnb_segs[k].second;
            gb.bn_c1[k] = gb.bn_c0[k] + st->tensors[bn.in].sh.C;
            gb.bn_z[k] = z.p;
            gb.ld_bnz[k] = z.ld;
            gb.bn_mean[k] = bst;
            gb.bn_rstd[k] = bst + bn.stat_ld;
          }
          int rb = 0;
          XP_HIP(launch_gap_bwd_bn(dt, pa, gb, s, &rb));
          st->bnb_nrb[i] = rb;
        }
        break;
      }
      case OP_CONCAT:
        break;
    }
    XP_OK(lanes.end(i, s));
  }
  return lanes.join();
}

// ---------------------------------------------------------------- coefficients
xpipe_status check_hp(const xpipe_hparams* hp) {
  if (!hp) return fail(XPIPE_EINVAL, "null hparams");
  if (!(hp->lr >= 0) || !(hp->beta1 >= 0 && hp->beta1 < 1) || !(hp->beta2 >= 0 && hp->beta2 < 1) ||
      !(hp->eps > 0) || hp->t < 0 || hp->mode < 0 || hp->mode > 3)
    return fail(XPIPE_EINVAL, "bad hparams");
  return XPIPE_OK;
}

PredCoef pred_coef(const xpipe_hparams* hp, int64_t t, int s) {
  PredCoef c{};
  c.eps = hp->eps;
  c.kind = hp->mode == XPIPE_PRED_ADAMDIR    ? PRED_DIR_ADAM
           : hp->mode == XPIPE_PRED_SMOOTHED ? PRED_DIR_SMOOTHED
                                             : PRED_DIR_EQ3;
  bool identity = s == 0 || (t == 0 && hp->mode != XPIPE_PRED_LITERAL);
  if (identity) return c;  // coef = c1 = c2 = 0: W - 0 * 0 = W
  c.coef = (double)s * hp->lr;
  if (hp->mode == XPIPE_PRED_SMOOTHED) {
    // the heavy-ball buffer of the same gradients, from the first moment
    c.c1 = 1.0 / (1.0 - hp->beta1);
  } else if (hp->mode == XPIPE_PRED_LITERAL) {
    c.c1 = 1.0 / (1.0 - hp->beta1);
    c.c2 = 1.0 / (1.0 - hp->beta2);
  } else {
    c.c1 = 1.0 / (1.0 - std::pow(hp->beta1, (double)t));
    c.c2 = 1.0 / (1.0 - std::pow(hp->beta2, (double)t));
  }
  return c;
}

AdamCoef adam_coef(const xpipe_hparams* hp) {
  AdamCoef a{};
  double t = (double)(hp->t + 1);
  a.lr = hp->lr;
  a.beta1 = hp->beta1;
  a.beta2 = hp->beta2;
  a.one_m_beta1 = 1.0 - hp->beta1;
  a.one_m_beta2 = 1.0 - hp->beta2;
  a.bc1 = 1.0 / (1.0 - std::pow(hp->beta1, t));
  a.bc2 = 1.0 / (1.0 - std::pow(hp->beta2, t));
  a.eps = hp->eps;
  return a;
}

xpipe_status check_rule(const xpipe_rule_hparams* rp) {
  if (!rp) return fail(XPIPE_EINVAL, "null rule hparams");
  if (rp->rule != XPIPE_RULE_MOMENTUM_SGD && rp->rule != XPIPE_RULE_RMSPROP)
    return fail(XPIPE_EINVAL, "unknown update rule");
  if (!(rp->lr >= 0) || !(rp->momentum >= 0 && rp->momentum < 1) || !(rp->weight_decay >= 0))
    return fail(XPIPE_EINVAL, "bad rule hparams");
  if (rp->rule == XPIPE_RULE_RMSPROP && (!(rp->alpha >= 0 && rp->alpha < 1) || !(rp->eps > 0)))
    return fail(XPIPE_EINVAL, "bad RMSProp hparams");
  return XPIPE_OK;
}

RuleCoef rule_coef(const xpipe_rule_hparams* rp, const xpipe_hparams* hp) {
  RuleCoef c{};
  c.lr = rp->lr;
  c.mu = rp->momentum;
  c.wd = rp->weight_decay;
  c.alpha = rp->alpha;
  c.one_m_alpha = 1.0 - rp->alpha;
  c.eps = rp->eps;
  c.beta1 = hp->beta1;
  c.beta2 = hp->beta2;
  c.one_m_beta1 = 1.0 - hp->beta1;
  c.one_m_beta2 = 1.0 - hp->beta2;
  return c;
}

// the merged GEMMs' weights, gathered from the prediction of direction dir
xpipe_status refresh_gathered(xpipe_stage* st, int dir) {
  // every merged GEMM's sibling weights, up to GATHER_BATCH copies per launch
  const size_t esz = st->esz();
  GatherArgs g{};
  for (const Op& op : st->ops) {
    if (op.segs.empty()) continue;
    const int64_t K = (int64_t)op.k * op.kw * op.cin;
    int64_t base = 0;
    for (const auto& sg : op.segs) {
      const int q = g.nseg++;
      if (st->dtype == DT_BF16)
        g.src[q] = st->wws + (dir == XPIPE_FWD ? st->bf_f_off : st->bf_b_off) + (size_t)sg.first * 2;
      else
        g.src[q] = (dir == XPIPE_FWD ? st->wpf : st->wpb) + sg.first;
      g.dst[q] = st->wws + op.wg_off[dir] + (size_t)base * esz;
      g.count[q] = K * sg.second;
      base += g.count[q];
      if (g.nseg == GATHER_BATCH) {
        XP_HIP(launch_gather(st->dtype, g, st->stream));
        g.nseg = 0;
      }
    }
  }
  if (g.nseg > 0) XP_HIP(launch_gather(st->dtype, g, st->stream));
  return XPIPE_OK;
}

xpipe_status refresh_flipped(xpipe_stage* st) {
  // same grid: flipped (the data gradient is a convolution of dy); strided or
  // unpadded: transposed only (the data gradient gathers dy tap by tap).  Up
  // to FLIP_MAX convolutions per launch.
  FlipSet f{};
  for (const Op& op : st->ops) {
    if (op.kind != OP_GEMM) continue;
    const int q = f.n++;
    f.w[q] = gemm_weights(st, op, XPIPE_BWD);
    f.wd[q] = st->wws + op.wd_off;
    f.N[q] = op.cout;
    f.R[q] = op.k;
    f.S[q] = op.kw;
    f.C[q] = op.cin;
    f.flip[q] = !op.grid;
    if (f.n == FLIP_MAX) {
      XP_HIP(launch_flip_set(st->dtype, f, st->stream));
      f.n = 0;
    }
  }
  XP_HIP(launch_flip_set(st->dtype, f, st->stream));
  st->wd_valid = true;
  return XPIPE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

void drop_graphs(xpipe_stage* st) {
  for (auto& g : st->pass_graphs) (void)hipGraphExecDestroy(g.exec);
  st->pass_graphs.clear();
}

// Forwards on their own stream (xpipe_stage_set_fwd_stream): a call that
// rewrites the forward prediction (or what derives from it) first makes the
// stage's stream wait for the forwards enqueued before it, and afterwards
// marks the point the next forward waits for.
xpipe_status wait_forwards(xpipe_stage* st) {
  if (!st->fwd_pending) return XPIPE_OK;
  XP_HIP(hipStreamWaitEvent(st->stream, st->fwd_ev, 0));
  st->fwd_pending = false;
  return XPIPE_OK;
}

xpipe_status mark_prediction(xpipe_stage* st) {
  if (!st->fwd_stream) return XPIPE_OK;
  XP_HIP(hipEventRecord(st->pred_ev, st->stream));
  return XPIPE_OK;
}

void release_lanes(xpipe_stage* st) {
  drop_graphs(st);
  if (st->pred_ev) (void)hipEventDestroy(st->pred_ev);
  if (st->fwd_ev) (void)hipEventDestroy(st->fwd_ev);
  if (st->cap_stream) (void)hipStreamDestroy(st->cap_stream);
  for (int pass = 0; pass < 2; ++pass)
    for (hipEvent_t e : st->op_ev[pass])
      if (e) (void)hipEventDestroy(e);
  if (st->fork_ev) (void)hipEventDestroy(st->fork_ev);
  for (int l = 1; l < NLANES; ++l) {
    if (st->join_ev[l]) (void)hipEventDestroy(st->join_ev[l]);
    if (st->lane_stream[l]) (void)hipStreamDestroy(st->lane_stream[l]);
  }
}

// Run one pass through its recorded graph: replay it if this (pass, pointers)
// was seen before, else capture the pass's launches on cap_stream (the lanes
// become graph edges), instantiate, keep, and replay.  The pass
// reads only the call's pointers and the stage's own buffers, so a recorded
// pass launches the same kernels with the same arguments as the eager one.
// Timing mode runs eagerly.
template <typename F>
xpipe_status run_graphed(xpipe_stage* st, int kind, const void* const (&ptr)[5], F&& pass) {
  if (!st->graphs || st->timing) return pass();
  ++st->graph_clock;
  for (auto& g : st->pass_graphs)
    if (g.kind == kind && std::equal(ptr, ptr + 5, g.ptr)) {
      g.used = st->graph_clock;
      XP_HIP(hipGraphLaunch(g.exec, st->stream));
      return XPIPE_OK;
    }
  hipStream_t caller = st->stream;
  st->stream = st->lane_stream[0] = st->cap_stream;
  st->capturing = true;
  hipError_t e = hipStreamBeginCapture(st->cap_stream, hipStreamCaptureModeThreadLocal);
  xpipe_status ps = e == hipSuccess ? pass() : XPIPE_OK;
  hipGraph_t graph = nullptr;
  hipError_t e2 = e == hipSuccess ? hipStreamEndCapture(st->cap_stream, &graph) : e;
  st->capturing = false;
  st->stream = st->lane_stream[0] = caller;
  if (ps != XPIPE_OK || e != hipSuccess || e2 != hipSuccess) {
    if (graph) (void)hipGraphDestroy(graph);
    if (ps != XPIPE_OK) return ps;
    return fail(XPIPE_EHIP, std::string("pass capture: ") + hipGetErrorString(e != hipSuccess ? e : e2));
  }
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (e != hipSuccess) return fail(XPIPE_EHIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(e));
  constexpr size_t MAX_GRAPHS = 64;
  if (st->pass_graphs.size() >= MAX_GRAPHS) {
    // the evicted graph may still run on either stream
    if (st->fwd_stream) XP_HIP(hipStreamSynchronize(st->fwd_stream));
    XP_HIP(hipStreamSynchronize(st->own_stream));
    auto old = std::min_element(st->pass_graphs.begin(), st->pass_graphs.end(),
                                [](const auto& a, const auto& b) { return a.used < b.used; });
    (void)hipGraphExecDestroy(old->exec);
    st->pass_graphs.erase(old);
  }
  xpipe_stage::PassGraph g{};
  g.kind = kind;
  std::copy(ptr, ptr + 5, g.ptr);
  g.exec = exec;
  g.used = st->graph_clock;
  st->pass_graphs.push_back(g);
  XP_HIP(hipGraphLaunch(exec, st->stream));
  return XPIPE_OK;
}

// ---------------------------------------------------------------- static workspace
// Workspace of the stages made by xpipe_stage_create_static: a file-scope
// device array (each GPU holds its own copy, at its own address, from the
// library's load until the process ends).  Host code never passes the array's
// name to a kernel or a copy -- on the host it is only a stand-in -- but the
// device address that hipGetSymbolAddress resolved, once per device, with that
// device current.  At most one such stage is alive per device: a stage keeps
// state in its workspace between calls (bf16 copies of the predictions, the
// data gradient's flipped weights), which a second stage would overwrite.
constexpr size_t XP_STATIC_WS_BYTES = XPIPE_STATIC_WORKSPACE_BYTES;
static __device__ __align__(256) unsigned char scratch[XP_STATIC_WS_BYTES];

struct StaticWs {
  bool resolved = false;
  void* ptr = nullptr;
  const xpipe_stage* owner = nullptr;
};
constexpr int XP_MAX_DEVICES = 64;
std::mutex g_static_mu;
StaticWs g_static_ws[XP_MAX_DEVICES];

// the current device's copy of the array (resolved on the first call on that
// device); call with g_static_mu held
xpipe_status static_workspace(int dev, void** ptr) {
  if (dev < 0 || dev >= XP_MAX_DEVICES) return fail(XPIPE_EUNSUPPORTED, "device index out of range");
  StaticWs& w = g_static_ws[dev];
  if (!w.resolved) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(XPIPE_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    w.ptr = p;
    w.resolved = true;
  }
  *ptr = w.ptr;
  return XPIPE_OK;
}

// grad = 0 with a kernel (no memset node if a caller records the stream)
__global__ __launch_bounds__(256) void k_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.f;
}

hipError_t zero_f32(float* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

// Shared body of xpipe_stage_create and xpipe_stage_create_static.
xpipe_status create_stage(const xpipe_layer_desc* layers, int32_t n_layers, int32_t micro_batch, int32_t T,
                          int32_t H, int32_t W, int32_t C, int32_t dtype, void* hip_stream, float* W_,
                          float* m, float* v, float* grad, float* w_pred_fwd, float* w_pred_bwd,
                          void* workspace, size_t workspace_bytes, int static_dev, xpipe_stage_t* out) {
  if (!out) return fail(XPIPE_EINVAL, "null output handle");
  *out = nullptr;
  if (T < 1) return fail(XPIPE_EINVAL, "T must be >= 1");
  Plan p;
  xpipe_status s = build_plan(layers, n_layers, micro_batch, H, W, C, dtype, p);
  if (s != XPIPE_OK) return s;
  if (p.P > 0 && (!W_ || !m || !v || !grad || !w_pred_fwd || !w_pred_bwd))
    return fail(XPIPE_EINVAL, "null device buffer");
  if (static_dev >= 0 && p.ws > XP_STATIC_WS_BYTES)
    return fail(XPIPE_EINVAL, "stage needs a workspace of " + std::to_string(p.ws) +
                                  " bytes, more than the static workspace's " +
                                  std::to_string(XP_STATIC_WS_BYTES) + " (use xpipe_stage_create)");
  if (!workspace) return fail(XPIPE_EINVAL, "null workspace");
  if (workspace_bytes < p.ws) return fail(XPIPE_EINVAL, "workspace too small");
  if ((reinterpret_cast<uintptr_t>(workspace) % WS_ALIGN) != 0)
    return fail(XPIPE_EINVAL, "workspace must be 256-byte aligned");
  if (!aligned16(W_) || !aligned16(m) || !aligned16(v) || !aligned16(grad) ||
      !aligned16(w_pred_fwd) || !aligned16(w_pred_bwd))
    return fail(XPIPE_EINVAL, "parameter buffers must be 16-byte aligned");
  xpipe_stage* st = new (std::nothrow) xpipe_stage();
  if (!st) return fail(XPIPE_EINVAL, "out of host memory");
  st->layers.assign(layers, layers + n_layers);
  st->mb = micro_batch;
  st->T = T;
  st->dtype = dtype;
  st->in_shape = Shape{micro_batch, H, W, C};
  st->stream = st->own_stream = (hipStream_t)hip_stream;
  st->W = W_;
  st->m = m;
  st->v = v;
  st->grad = grad;
  st->wpf = w_pred_fwd;
  st->wpb = w_pred_bwd;
  st->ws = st->wws = (char*)workspace;
  st->ws_bytes = workspace_bytes;
  st->ws_need = p.ws;
  st->P = p.P;
  st->params = p.params;
  st->tensors = p.tensors;
  st->ops = p.ops;
  st->bnb_nrb.assign(st->ops.size(), 0);
  st->rec_order[0] = p.rec_order[0];
  st->rec_order[1] = p.rec_order[1];
  st->apply_groups = p.apply_groups;
  st->out_tensor = p.out_tensor;
  st->has_loss = p.has_loss;
  st->classes = p.classes;
  st->bf_f_off = p.bf_f_off;
  st->bf_b_off = p.bf_b_off;
  for (int l = 0; l < NLANES; ++l) {
    st->colpart_off[l] = p.colpart_off[l];
    st->wpart_off[l] = p.wpart_off[l];
  }
  st->hook.st = st;
  st->lane_stream[0] = st->stream;
  hipError_t e = hipSuccess;
  if (static_dev >= 0) {
    // everything on the caller's stream: no streams, events or graphs to create
    st->one_lane = true;
    st->graphs = false;
    st->static_dev = static_dev;
  } else {
    // auxiliary launch lanes (default priority) and their events
    for (int l = 1; l < NLANES && e == hipSuccess; ++l)
      e = hipStreamCreateWithFlags(&st->lane_stream[l], hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&st->cap_stream, hipStreamNonBlocking);
    if (const char* g = std::getenv("XPIPE_GRAPHS"); g && *g == '0') st->graphs = false;
    if (e == hipSuccess) e = hipEventCreateWithFlags(&st->fork_ev, hipEventDisableTiming);
    for (int l = 1; l < NLANES && e == hipSuccess; ++l)
      e = hipEventCreateWithFlags(&st->join_ev[l], hipEventDisableTiming);
    for (int pass = 0; pass < 2 && e == hipSuccess; ++pass) {
      st->op_ev[pass].assign(st->ops.size(), nullptr);
      for (size_t i = 0; i < st->ops.size() && e == hipSuccess; ++i)
        if (st->ops[i].record[pass])
          e = hipEventCreateWithFlags(&st->op_ev[pass][i], hipEventDisableTiming);
    }
    if (e != hipSuccess) {
      release_lanes(st);
      delete st;
      return fail(XPIPE_EHIP, std::string("stream / event creation: ") + hipGetErrorString(e));
    }
  }
  e = zero_f32(grad, p.P, st->stream);
  if (e != hipSuccess) {
    release_lanes(st);
    delete st;
    return fail(XPIPE_EHIP, std::string("zeroing grad: ") + hipGetErrorString(e));
  }
  *out = st;
  return XPIPE_OK;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================
extern "C" {

const char* xpipe_last_error(void) { return g_err.c_str(); }

static int round_rule(double x, int rule) {
  double lo = std::floor(x);
  double frac = x - lo;
  if (frac > 0.5) return (int)lo + 1;
  if (frac < 0.5) return (int)lo;
  if (rule == XPIPE_ROUND_HALF_UP) return (int)lo + 1;
  if (rule == XPIPE_ROUND_HALF_DOWN) return (int)lo;
  return ((int64_t)lo % 2 == 0) ? (int)lo : (int)lo + 1;
}

xpipe_status xpipe_version_difference(int32_t size, int32_t T, int32_t rank, int32_t dir,
                                      int32_t rounding, int32_t ceil_half_rank, int32_t* s_out) {
  if (!s_out) return fail(XPIPE_EINVAL, "null output");
  if (size < 1 || T < 1 || rank < 0 || rank >= size) return fail(XPIPE_EINVAL, "need size >= 1, T >= 1, 0 <= rank < size");
  if (dir != XPIPE_FWD && dir != XPIPE_BWD) return fail(XPIPE_EINVAL, "bad direction");
  if (rounding < 0 || rounding > 2) return fail(XPIPE_EINVAL, "bad rounding rule");
  double x;
  if (dir == XPIPE_FWD) {
    double half = ceil_half_rank ? (double)((rank + 1) / 2) : rank / 2.0;
    x = ((double)size + T - half - 2.0) / T;
  } else {
    x = ((double)T + rank / 2 - 1.0) / T;
  }
  *s_out = round_rule(x, rounding);
  return XPIPE_OK;
}

xpipe_status xpipe_stage_query(const xpipe_layer_desc* layers, int32_t n_layers, int32_t micro_batch,
                               int32_t H, int32_t W, int32_t C, int32_t dtype,
                               int64_t* n_params_padded, size_t* workspace_bytes) {
  if (!n_params_padded || !workspace_bytes) return fail(XPIPE_EINVAL, "null output");
  Plan p;
  xpipe_status s = build_plan(layers, n_layers, micro_batch, H, W, C, dtype, p);
  if (s != XPIPE_OK) return s;
  *n_params_padded = p.P;
  *workspace_bytes = p.ws;
  return XPIPE_OK;
}

xpipe_status xpipe_stage_create(const xpipe_layer_desc* layers, int32_t n_layers, int32_t micro_batch,
                                int32_t T, int32_t H, int32_t W, int32_t C, int32_t dtype,
                                void* hip_stream, float* W_, float* m, float* v, float* grad,
                                float* w_pred_fwd, float* w_pred_bwd, void* workspace,
                                size_t workspace_bytes, xpipe_stage_t* out) {
  return create_stage(layers, n_layers, micro_batch, T, H, W, C, dtype, hip_stream, W_, m, v, grad,
                      w_pred_fwd, w_pred_bwd, workspace, workspace_bytes, -1, out);
}

xpipe_status xpipe_stage_create_static(const xpipe_layer_desc* layers, int32_t n_layers,
                                       int32_t micro_batch, int32_t T, int32_t H, int32_t W, int32_t C,
                                       int32_t dtype, void* hip_stream, float* W_, float* m, float* v,
                                       float* grad, float* w_pred_fwd, float* w_pred_bwd,
                                       xpipe_stage_t* out) {
  if (!out) return fail(XPIPE_EINVAL, "null output handle");
  *out = nullptr;
  int dev = -1;
  XP_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(g_static_mu);
  void* ws = nullptr;
  xpipe_status s = static_workspace(dev, &ws);
  if (s != XPIPE_OK) return s;
  if (g_static_ws[dev].owner)
    return fail(XPIPE_ESTATE, "a stage with the static workspace is alive on this device "
                              "(destroy it first)");
  s = create_stage(layers, n_layers, micro_batch, T, H, W, C, dtype, hip_stream, W_, m, v, grad,
                   w_pred_fwd, w_pred_bwd, ws, XP_STATIC_WS_BYTES, dev, out);
  if (s == XPIPE_OK) g_static_ws[dev].owner = *out;
  return s;
}

xpipe_status xpipe_stage_num_param_tensors(xpipe_stage_t st, int32_t* n) {
  if (!st || !n) return fail(XPIPE_EINVAL, "null argument");
  *n = (int32_t)st->params.size();
  return XPIPE_OK;
}

xpipe_status xpipe_stage_param_layout(xpipe_stage_t st, int32_t idx, int64_t* offset, int64_t* count) {
  if (!st || !offset || !count) return fail(XPIPE_EINVAL, "null argument");
  if (idx < 0 || idx >= (int32_t)st->params.size()) return fail(XPIPE_EINVAL, "tensor index out of range");
  *offset = st->params[idx].off;
  *count = st->params[idx].count;
  return XPIPE_OK;
}

xpipe_status xpipe_stage_output_shape(xpipe_stage_t st, int32_t* n, int32_t* H, int32_t* W, int32_t* C) {
  if (!st || !n || !H || !W || !C) return fail(XPIPE_EINVAL, "null argument");
  const Shape& s = st->tensors[st->out_tensor].sh;
  *n = s.n;
  *H = s.H;
  *W = s.W;
  *C = s.C;
  return XPIPE_OK;
}

xpipe_status xpipe_predict_weights(xpipe_stage_t st, int32_t which, int32_t s, const xpipe_hparams* hp) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (which != XPIPE_FWD && which != XPIPE_BWD) return fail(XPIPE_EINVAL, "bad direction");
  if (s < 0) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  HookScope hs_(st);
  PredCoef c = pred_coef(hp, hp->t, s);
  float* out = which == XPIPE_FWD ? st->wpf : st->wpb;
  bf16_t* obf = nullptr;
  if (st->dtype == DT_BF16) obf = (bf16_t*)(st->wws + (which == XPIPE_FWD ? st->bf_f_off : st->bf_b_off));
  if (which == XPIPE_FWD) XP_OK(wait_forwards(st));
  {
    XP_HIP(launch_predict(st->W, st->m, st->v, out, obf, st->P, c, st->stream));
  }
  xpipe_status r = refresh_gathered(st, which);
  if (r != XPIPE_OK) return r;
  st->pred_valid[which] = true;
  if (which == XPIPE_BWD) {
    r = refresh_flipped(st);
    if (r != XPIPE_OK) return r;
    return XPIPE_OK;
  }
  return mark_prediction(st);
}

xpipe_status xpipe_stage_fwd(xpipe_stage_t st, const void* x, void* y, const int32_t* labels, float* loss) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (!x || !y) return fail(XPIPE_EINVAL, "null input or output");
  if (st->has_loss && loss && !labels) return fail(XPIPE_EINVAL, "labels required for the loss");
  if (!st->pred_valid[XPIPE_FWD]) return fail(XPIPE_ESTATE, "no forward prediction: call xpipe_predict_weights(FWD) first");
  HookScope hs_(st);
  Ctx c;
  c.x = x;
  c.y = y;
  float* ls = st->has_loss ? loss : nullptr;
  const void* const key[5] = {x, y, labels, ls, nullptr};
  // (timing mode: on the stage's stream, but the same launches)
  if (!st->fwd_stream || st->timing)
    return run_graphed(st, 0, key,
                       [&] { return run_forward(st, XPIPE_FWD, c, labels, ls, st->fwd_stream != nullptr); });
  // on the forward stream, with the forward workspace, after the last write
  // of the forward prediction
  XP_HIP(hipStreamWaitEvent(st->fwd_stream, st->pred_ev, 0));
  hipStream_t caller = st->stream;
  char* pass_ws = st->ws;
  st->stream = st->lane_stream[0] = st->fwd_stream;
  st->ws = st->fwd_ws;
  // one chain of launches (no auxiliary lanes), as is the recomputed forward
  // of the backwards beside it: on the Inception-A step 6.28 ms against 6.35
  // with both on the forward's three lanes (6.50 with only this forward
  // chained, 6.65 with only the recomputed one)
  xpipe_status r = run_graphed(st, 0, key, [&] { return run_forward(st, XPIPE_FWD, c, labels, ls, true); });
  st->stream = st->lane_stream[0] = caller;
  st->ws = pass_ws;
  if (r != XPIPE_OK) return r;
  XP_HIP(hipEventRecord(st->fwd_ev, st->fwd_stream));
  st->fwd_pending = true;
  return XPIPE_OK;
}

xpipe_status xpipe_stage_bwd(xpipe_stage_t st, const void* x, const void* dy, const int32_t* labels, void* dx) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (!x) return fail(XPIPE_EINVAL, "null input");
  if (st->has_loss && !labels) return fail(XPIPE_EINVAL, "labels required for a loss stage");
  if (!st->has_loss && !dy) return fail(XPIPE_EINVAL, "dy required for a stage without a loss");
  if (!st->pred_valid[XPIPE_BWD] || !st->wd_valid)
    return fail(XPIPE_ESTATE, "no backward prediction: call xpipe_predict_weights(BWD) first");
  HookScope hs_(st);
  Ctx c;
  c.x = x;
  c.dx = dx;
  const void* const key[5] = {x, dy, labels, dx, nullptr};
  xpipe_status s = run_graphed(st, 1, key, [&] {
    // with the forwards on their own stream, the recomputed forward is one
    // chain too (see xpipe_stage_fwd)
    xpipe_status r = run_forward(st, XPIPE_BWD, c, nullptr, nullptr, st->fwd_stream != nullptr);
    return r != XPIPE_OK ? r : run_backward(st, c, dy, labels);
  });
  if (s != XPIPE_OK) return s;
  st->bwd_since_step++;
  return XPIPE_OK;
}

xpipe_status xpipe_stage_set_fwd_stream(xpipe_stage_t st, void* workspace, size_t workspace_bytes,
                                        void** hip_stream) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (hip_stream) *hip_stream = nullptr;
  if (workspace) {
    if (st->one_lane) return fail(XPIPE_EUNSUPPORTED, "a static-workspace stage runs on one stream");
    if (workspace_bytes < st->ws_need) return fail(XPIPE_EINVAL, "forward workspace too small");
    if ((reinterpret_cast<uintptr_t>(workspace) % WS_ALIGN) != 0)
      return fail(XPIPE_EINVAL, "forward workspace must be 256-byte aligned");
  }
  // the recorded forwards used the other workspace and stream: finish them
  if (st->fwd_stream) XP_HIP(hipStreamSynchronize(st->fwd_stream));
  XP_HIP(hipStreamSynchronize(st->stream));
  st->fwd_pending = false;
  drop_graphs(st);
  // The stage's last launch lane, which no pass uses while the forwards have
  // their own stream (the forward and the recomputed forward are chains on
  // lane 0, the backward starts chains on PASS_LANES[1] lanes).  Measured
  // against a stream of the caller's (torch's stream pool): the same step
  // times when the two streams land on different hardware queues, but from
  // one stage creation to the next the caller's stream could share the
  // stage's queue (VGG stage 0.98 against 0.86 ms, ResNet middle stage 7.31
  // against 6.41 ms, Inception-A 7.82 against 6.29 ms); the lane was 0.86,
  // 6.40-6.41 and 6.28-6.35 ms every time.  A stream with a hardware queue of
  // its own (a full CU mask) was 1.3-5x slower.
  static_assert(PASS_LANES[1] < NLANES, "the forward stream is a lane the backward does not use");
  hipStream_t fs = workspace ? st->lane_stream[NLANES - 1] : nullptr;
  st->fwd_stream = fs;
  st->fwd_ws = fs ? (char*)workspace : nullptr;
  if (!fs) return XPIPE_OK;
  if (!st->pred_ev) XP_HIP(hipEventCreateWithFlags(&st->pred_ev, hipEventDisableTiming));
  if (!st->fwd_ev) XP_HIP(hipEventCreateWithFlags(&st->fwd_ev, hipEventDisableTiming));
  XP_HIP(hipEventRecord(st->pred_ev, st->stream));
  if (hip_stream) *hip_stream = (void*)fs;
  return XPIPE_OK;
}

xpipe_status xpipe_stage_set_graphs(xpipe_stage_t st, int32_t enable) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (st->one_lane && enable) return fail(XPIPE_EUNSUPPORTED, "a static-workspace stage records no passes");
  // the kept graphs may still run
  if (st->fwd_stream) XP_HIP(hipStreamSynchronize(st->fwd_stream));
  XP_HIP(hipStreamSynchronize(st->stream));
  st->graphs = enable != 0;
  drop_graphs(st);
  return XPIPE_OK;
}

xpipe_status xpipe_adam_step(xpipe_stage_t st, const xpipe_hparams* hp, int32_t s_fwd_next,
                             int32_t s_bwd_next, int32_t emit_pred) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  const bool keep = emit_pred == XPIPE_KEEP_PRED;
  if (keep) emit_pred = 0;
  if (emit_pred && (s_fwd_next < 0 || s_bwd_next < 0)) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  if (st->bwd_since_step == 0) return fail(XPIPE_ESTATE, "no backward since the last update");
  HookScope hs_(st);
  AdamCoef a = adam_coef(hp);
  PredCoef cf = pred_coef(hp, hp->t + 1, s_fwd_next);
  PredCoef cb = pred_coef(hp, hp->t + 1, s_bwd_next);
  bf16_t* ff = nullptr;
  bf16_t* fb = nullptr;
  if (emit_pred && st->dtype == DT_BF16) {
    ff = (bf16_t*)(st->wws + st->bf_f_off);
    fb = (bf16_t*)(st->wws + st->bf_b_off);
  }
  if (emit_pred) XP_OK(wait_forwards(st));
  {
    XP_HIP(launch_adam(st->W, st->m, st->v, st->grad, st->P, a, 1, emit_pred ? st->wpf : nullptr, ff, cf,
                       emit_pred ? st->wpb : nullptr, fb, cb, st->stream));
  }
  st->bwd_since_step = 0;
  if (keep) return XPIPE_OK;  // the cached predictions (and what derives from them) stay
  st->pred_valid[0] = st->pred_valid[1] = emit_pred != 0;
  st->wd_valid = false;
  if (!emit_pred) return XPIPE_OK;
  for (int d = 0; d < 2; ++d) {
    xpipe_status r = refresh_gathered(st, d);
    if (r != XPIPE_OK) return r;
  }
  XP_OK(refresh_flipped(st));
  return mark_prediction(st);
}

xpipe_status xpipe_rule_step(xpipe_stage_t st, const xpipe_rule_hparams* rp, const xpipe_hparams* hp,
                             float* buf, float* sq, int32_t s_fwd_next, int32_t s_bwd_next,
                             int32_t emit_pred) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  hs = check_rule(rp);
  if (hs != XPIPE_OK) return hs;
  const bool keep = emit_pred == XPIPE_KEEP_PRED;
  if (keep) emit_pred = 0;
  if (emit_pred && (s_fwd_next < 0 || s_bwd_next < 0)) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  if (!buf || (rp->rule == XPIPE_RULE_RMSPROP && !sq)) return fail(XPIPE_EINVAL, "null optimizer buffer");
  if (!aligned16(buf) || (sq && !aligned16(sq))) return fail(XPIPE_EINVAL, "buffers must be 16-byte aligned");
  if (st->bwd_since_step == 0) return fail(XPIPE_ESTATE, "no backward since the last update");
  HookScope hs_(st);
  PredCoef cf = pred_coef(hp, hp->t + 1, s_fwd_next);
  PredCoef cb = pred_coef(hp, hp->t + 1, s_bwd_next);
  bf16_t* ff = nullptr;
  bf16_t* fb = nullptr;
  if (emit_pred && st->dtype == DT_BF16) {
    ff = (bf16_t*)(st->wws + st->bf_f_off);
    fb = (bf16_t*)(st->wws + st->bf_b_off);
  }
  if (emit_pred) XP_OK(wait_forwards(st));
  XP_HIP(launch_rule(rp->rule, st->W, buf, sq, st->m, st->v, st->grad, st->P, rule_coef(rp, hp), 1,
                     emit_pred ? st->wpf : nullptr, ff, cf, emit_pred ? st->wpb : nullptr, fb, cb, st->stream));
  st->bwd_since_step = 0;
  if (keep) return XPIPE_OK;
  st->pred_valid[0] = st->pred_valid[1] = emit_pred != 0;
  st->wd_valid = false;
  if (!emit_pred) return XPIPE_OK;
  for (int d = 0; d < 2; ++d) {
    xpipe_status r = refresh_gathered(st, d);
    if (r != XPIPE_OK) return r;
  }
  XP_OK(refresh_flipped(st));
  return mark_prediction(st);
}

xpipe_status xpipe_stage_destroy(xpipe_stage_t st) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  // auxiliary lanes (and the forward stream) finish their work before the
  // streams, events and graphs go away
  if (st->fwd_stream) (void)hipStreamSynchronize(st->fwd_stream);
  for (int l = 1; l < NLANES; ++l)
    if (st->lane_stream[l]) (void)hipStreamSynchronize(st->lane_stream[l]);
  release_lanes(st);
  for (auto& r : st->pending) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : st->pool) (void)hipEventDestroy(e);
  if (st->static_dev >= 0) {
    // work still queued on the caller's stream uses the static workspace
    (void)hipStreamSynchronize(st->stream);
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (g_static_ws[st->static_dev].owner == st) g_static_ws[st->static_dev].owner = nullptr;
  }
  delete st;
  return XPIPE_OK;
}

xpipe_status xpipe_predict_flat(const float* W, const float* m, const float* v, float* out, uint16_t* out_bf16,
                                int64_t n, int32_t s, const xpipe_hparams* hp, void* hip_stream) {
  if (n < 0) return fail(XPIPE_EINVAL, "negative length");
  if (s < 0) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  if (n == 0) return XPIPE_OK;
  if (!W || !m || !v || !out) return fail(XPIPE_EINVAL, "null buffer");
  if (!aligned16(W) || !aligned16(m) || !aligned16(v) || !aligned16(out) ||
      (out_bf16 && (reinterpret_cast<uintptr_t>(out_bf16) & 7) != 0))
    return fail(XPIPE_EINVAL, "buffers must be 16-byte aligned (bf16 output 8-byte)");
  XP_HIP(launch_predict(W, m, v, out, out_bf16, n, pred_coef(hp, hp->t, s), (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_adam_flat(float* W, float* m, float* v, float* G, int64_t n, const xpipe_hparams* hp,
                             int32_t zero_grad, float* pred_fwd, int32_t s_fwd, float* pred_bwd, int32_t s_bwd,
                             void* hip_stream) {
  if (n < 0) return fail(XPIPE_EINVAL, "negative length");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  if ((pred_fwd && s_fwd < 0) || (pred_bwd && s_bwd < 0)) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  if (n == 0) return XPIPE_OK;
  if (!W || !m || !v || !G) return fail(XPIPE_EINVAL, "null buffer");
  if (!aligned16(W) || !aligned16(m) || !aligned16(v) || !aligned16(G) ||
      (pred_fwd && !aligned16(pred_fwd)) || (pred_bwd && !aligned16(pred_bwd)))
    return fail(XPIPE_EINVAL, "buffers must be 16-byte aligned");
  XP_HIP(launch_adam(W, m, v, G, n, adam_coef(hp), zero_grad, pred_fwd, nullptr, pred_coef(hp, hp->t + 1, s_fwd),
                     pred_bwd, nullptr, pred_coef(hp, hp->t + 1, s_bwd), (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_rule_flat(float* W, float* buf, float* sq, float* m, float* v, float* G, int64_t n,
                             const xpipe_rule_hparams* rp, const xpipe_hparams* hp, int32_t zero_grad,
                             float* pred_fwd, int32_t s_fwd, float* pred_bwd, int32_t s_bwd,
                             void* hip_stream) {
  if (n < 0) return fail(XPIPE_EINVAL, "negative length");
  xpipe_status hs = check_hp(hp);
  if (hs != XPIPE_OK) return hs;
  hs = check_rule(rp);
  if (hs != XPIPE_OK) return hs;
  if ((pred_fwd && s_fwd < 0) || (pred_bwd && s_bwd < 0)) return fail(XPIPE_EINVAL, "version difference must be >= 0");
  if (n == 0) return XPIPE_OK;
  if (!W || !buf || !m || !v || !G || (rp->rule == XPIPE_RULE_RMSPROP && !sq)) return fail(XPIPE_EINVAL, "null buffer");
  if (!aligned16(W) || !aligned16(buf) || (sq && !aligned16(sq)) || !aligned16(m) || !aligned16(v) ||
      !aligned16(G) || (pred_fwd && !aligned16(pred_fwd)) || (pred_bwd && !aligned16(pred_bwd)))
    return fail(XPIPE_EINVAL, "buffers must be 16-byte aligned");
  XP_HIP(launch_rule(rp->rule, W, buf, sq, m, v, G, n, rule_coef(rp, hp), zero_grad, pred_fwd, nullptr,
                     pred_coef(hp, hp->t + 1, s_fwd), pred_bwd, nullptr, pred_coef(hp, hp->t + 1, s_bwd),
                     (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_probe_copy(const void* src, void* dst, int64_t bytes, void* hip_stream) {
  if (bytes < 0 || (bytes % 16) != 0) return fail(XPIPE_EINVAL, "bytes must be a multiple of 16");
  if (bytes == 0) return XPIPE_OK;
  if (!src || !dst) return fail(XPIPE_EINVAL, "null buffer");
  if (!aligned16(src) || !aligned16(dst)) return fail(XPIPE_EINVAL, "buffers must be 16-byte aligned");
  XP_HIP(launch_probe_copy(src, dst, bytes, (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_probe_stream(const float* const* src, int32_t nsrc, float* const* dst, int32_t ndst,
                                int64_t n, void* hip_stream) {
  if (n < 0 || (n % 4) != 0) return fail(XPIPE_EINVAL, "n must be a non-negative multiple of 4");
  if (nsrc < 0 || nsrc > STREAM_MAX_SRC || ndst < 1 || ndst > STREAM_MAX_DST)
    return fail(XPIPE_EINVAL, "0..4 sources and 1..6 destinations");
  if (n == 0) return XPIPE_OK;
  if ((nsrc > 0 && !src) || !dst) return fail(XPIPE_EINVAL, "null pointer array");
  StreamArgs a{};
  for (int j = 0; j < nsrc; ++j) {
    if (!src[j] || !aligned16(src[j])) return fail(XPIPE_EINVAL, "sources must be 16-byte aligned");
    a.src[j] = src[j];
  }
  for (int j = 0; j < ndst; ++j) {
    if (!dst[j] || !aligned16(dst[j])) return fail(XPIPE_EINVAL, "destinations must be 16-byte aligned");
    a.dst[j] = dst[j];
  }
  a.nsrc = nsrc;
  a.ndst = ndst;
  a.n = n / 4;
  XP_HIP(launch_probe_stream(a, (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_probe_mfma(float* out, int32_t waves, int32_t iters, void* hip_stream) {
  if (waves < 0 || iters < 0) return fail(XPIPE_EINVAL, "negative size");
  if (waves == 0 || iters == 0) return XPIPE_OK;
  if (!out) return fail(XPIPE_EINVAL, "null output");
  XP_HIP(launch_probe_mfma(out, waves, iters, (hipStream_t)hip_stream));
  return XPIPE_OK;
}

xpipe_status xpipe_probe_graph(float* scratch, int32_t width, int32_t len, int32_t reps, int32_t spin,
                               double* us_out, void* hip_stream) {
  if (!scratch || !us_out) return fail(XPIPE_EINVAL, "null pointer");
  if (width < 1 || width > 3 || len < 1 || len > 8 || reps < 1 || reps > 256 || spin < 0)
    return fail(XPIPE_EINVAL, "probe sizes out of range");
  // recorded and replayed on a stream of its own (a capture cannot use the
  // null stream), after the work already on hip_stream; returns when done
  hipStream_t s0 = nullptr;
  hipStream_t side[3] = {nullptr, nullptr, nullptr};
  std::vector<hipEvent_t> evs;
  hipGraph_t g = nullptr;
  hipGraphExec_t ge = nullptr;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  hipError_t e = hipSuccess;
  auto ev = [&](hipEvent_t* out) {
    e = hipEventCreateWithFlags(out, hipEventDisableTiming);
    if (e == hipSuccess) evs.push_back(*out);
    return e;
  };
  // one recorded graph per layout; the stream work happens while capturing
  auto record = [&](bool branches) -> hipError_t {
    hipError_t r = hipStreamBeginCapture(s0, hipStreamCaptureModeThreadLocal);
    if (r != hipSuccess) return r;
    int k = 0;
    for (int q = 0; q < reps && r == hipSuccess; ++q) {
      r = launch_probe_spin(scratch, k++, spin, 256, s0);
      if (r != hipSuccess || !branches) {
        for (int b = 0; b < width * len && r == hipSuccess; ++b) r = launch_probe_spin(scratch, k++, spin, 256, s0);
        continue;
      }
      hipEvent_t f;
      if ((r = ev(&f)) != hipSuccess || (r = hipEventRecord(f, s0)) != hipSuccess) break;
      for (int b = 0; b < width && r == hipSuccess; ++b) {
        if ((r = hipStreamWaitEvent(side[b], f, 0)) != hipSuccess) break;
        for (int l = 0; l < len && r == hipSuccess; ++l) r = launch_probe_spin(scratch, k++, spin, 256, side[b]);
        hipEvent_t j;
        if (r != hipSuccess || (r = ev(&j)) != hipSuccess || (r = hipEventRecord(j, side[b])) != hipSuccess) break;
        r = hipStreamWaitEvent(s0, j, 0);
      }
    }
    hipGraph_t gg = nullptr;
    hipError_t r2 = hipStreamEndCapture(s0, &gg);
    if (r == hipSuccess) r = r2;
    if (r == hipSuccess) g = gg;
    else if (gg) hipGraphDestroy(gg);
    return r;
  };
  for (int b = 0; b < width && e == hipSuccess; ++b) e = hipStreamCreateWithFlags(&side[b], hipStreamNonBlocking);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&s0, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreate(&t0);
  if (e == hipSuccess) e = hipEventCreate(&t1);
  if (e == hipSuccess) e = hipEventRecord(t0, (hipStream_t)hip_stream);
  if (e == hipSuccess) e = hipStreamWaitEvent(s0, t0, 0);
  for (int layout = 0; layout < 2 && e == hipSuccess; ++layout) {
    e = record(layout == 0);
    if (e == hipSuccess) e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    for (int w = 0; w < 2 && e == hipSuccess; ++w) e = hipGraphLaunch(ge, s0);
    if (e == hipSuccess) e = hipEventRecord(t0, s0);
    for (int w = 0; w < 5 && e == hipSuccess; ++w) e = hipGraphLaunch(ge, s0);
    if (e == hipSuccess) e = hipEventRecord(t1, s0);
    if (e == hipSuccess) e = hipEventSynchronize(t1);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, t0, t1);
    if (e == hipSuccess) us_out[layout] = (double)ms * 1e3 / 5.0 / reps;
    if (ge) hipGraphExecDestroy(ge);
    if (g) hipGraphDestroy(g);
    ge = nullptr;
    g = nullptr;
  }
  for (hipEvent_t x : evs) hipEventDestroy(x);
  if (t0) hipEventDestroy(t0);
  if (t1) hipEventDestroy(t1);
  if (s0) {
    hipStreamSynchronize(s0);
    hipStreamDestroy(s0);
  }
  for (int b = 0; b < 3; ++b)
    if (side[b]) hipStreamDestroy(side[b]);
  if (e != hipSuccess) return fail(XPIPE_EHIP, std::string("graph probe: ") + hipGetErrorString(e));
  return XPIPE_OK;
}

xpipe_status xpipe_stage_set_timing(xpipe_stage_t st, int32_t enable) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  st->timing = enable != 0;
  st->agg.clear();
  for (auto& r : st->pending) {
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
  }
  st->pending.clear();
  return XPIPE_OK;
}

static xpipe_status drain_timing(xpipe_stage* st) {
  for (auto& r : st->pending) {
    float e = 0.f;
    hipError_t err = hipEventSynchronize(r.b);
    if (err != hipSuccess) return fail(XPIPE_EHIP, std::string("hipEventSynchronize: ") + hipGetErrorString(err));
    err = hipEventElapsedTime(&e, r.a, r.b);
    if (err != hipSuccess) return fail(XPIPE_EHIP, std::string("hipEventElapsedTime: ") + hipGetErrorString(err));
    TimeAgg& g = st->agg[r.name];
    g.ms += e;
    g.work += r.work;
    g.n += 1;
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
  }
  st->pending.clear();
  return XPIPE_OK;
}

xpipe_status xpipe_stage_timing_count(xpipe_stage_t st, int32_t* n) {
  if (!st || !n) return fail(XPIPE_EINVAL, "null argument");
  xpipe_status s = drain_timing(st);
  if (s != XPIPE_OK) return s;
  *n = (int32_t)st->agg.size();
  return XPIPE_OK;
}

xpipe_status xpipe_stage_timing_entry(xpipe_stage_t st, int32_t i, const char** kernel, double* ms,
                                      int64_t* launches, double* work) {
  if (!st || !kernel || !ms || !launches || !work) return fail(XPIPE_EINVAL, "null argument");
  xpipe_status s = drain_timing(st);
  if (s != XPIPE_OK) return s;
  if (i < 0 || i >= (int32_t)st->agg.size()) return fail(XPIPE_EINVAL, "timing entry out of range");
  auto it = st->agg.begin();
  std::advance(it, i);
  *kernel = it->first.c_str();
  *ms = it->second.ms;
  *launches = it->second.n;
  *work = it->second.work;
  return XPIPE_OK;
}

}  // extern "C"

// ============================================================================
// Pipeline schedule (unit-time model, Sec. III-A) and the interleaved executor
// ============================================================================
xpipe_status xpipe_schedule(int32_t size, int32_t T, int32_t rank, int32_t minibatches, int32_t rounding,
                            int32_t ceil_half_rank, xpipe_sched_event* out, int32_t capacity,
                            int32_t* count) {
  if (!count) return fail(XPIPE_EINVAL, "null output");
  if (size < 1 || T < 1 || rank < 0 || rank >= size || minibatches < 0)
    return fail(XPIPE_EINVAL, "need size >= 1, T >= 1, 0 <= rank < size, minibatches >= 0");
  if ((int64_t)T * minibatches > (1 << 28)) return fail(XPIPE_EINVAL, "schedule too long");
  const int32_t n = T * minibatches;
  *count = 2 * n;
  if (!out) return XPIPE_OK;
  if (capacity < 2 * n) return fail(XPIPE_EINVAL, "capacity below the event count");
  int32_t s_fwd = 0, s_bwd = 0;
  xpipe_status st = xpipe_version_difference(size, T, rank, XPIPE_FWD, rounding, ceil_half_rank, &s_fwd);
  if (st != XPIPE_OK) return st;
  st = xpipe_version_difference(size, T, rank, XPIPE_BWD, rounding, ceil_half_rank, &s_bwd);
  if (st != XPIPE_OK) return st;
  const int64_t K = size;
  auto fwd_time = [&](int64_t i) { return 2 * i + rank; };
  auto bwd_time = [&](int64_t i, int64_t r) { return 2 * i + 2 * K - 1 - r; };
  // forward and backward units have opposite parity, so the two ascending
  // sequences merge without ties; the updates are the backward units of the
  // T-th micro-batches, in ascending order
  int64_t f = 1, b = 1, updates_before = 0;
  for (int32_t q = 0; q < 2 * n; ++q) {
    const bool take_f = f <= n && (b > n || fwd_time(f) < bwd_time(b, rank));
    const int64_t i = take_f ? f++ : b++;
    const int64_t time = take_f ? fwd_time(i) : bwd_time(i, rank);
    // updates strictly before this unit
    while (updates_before < minibatches && bwd_time(T * (updates_before + 1), rank) < time) ++updates_before;
    xpipe_sched_event e{};
    e.time = (int32_t)time;
    e.kind = take_f ? XPIPE_FWD : XPIPE_BWD;
    e.micro = (int32_t)i;
    e.mini = (int32_t)((i - 1) / T + 1);
    e.bellwether = (i - 1) % T == 0;
    e.update_after = !take_f && i % T == 0;
    e.version = (int32_t)updates_before;
    if (e.bellwether) {
      e.s_eq = take_f ? s_fwd : s_bwd;
      const int64_t end = bwd_time((int64_t)T * e.mini, 0);     // round trip ends on GPU 0
      const int64_t own = bwd_time((int64_t)T * e.mini, rank);  // this mini-batch's update here
      int32_t incl = 0, excl = 0;
      for (int64_t j = 1; j <= minibatches; ++j) {
        const int64_t u = bwd_time(T * j, rank);
        if (u > time && u <= end) {
          ++incl;
          if (u != own) ++excl;
        }
      }
      e.s_incl = incl;
      e.s_excl = excl;
    }
    out[q] = e;
  }
  return XPIPE_OK;
}

xpipe_status xpipe_stage_run(xpipe_stage_t st, const xpipe_sched_event* events, int32_t n_events,
                             const xpipe_run_io* io, const xpipe_hparams* hp,
                             const xpipe_rule_hparams* rule, float* buf, float* sq, int32_t draft) {
  if (!st) return fail(XPIPE_EINVAL, "null stage");
  if (n_events < 0 || (n_events > 0 && !events)) return fail(XPIPE_EINVAL, "bad event list");
  if (!io || !io->x || !io->y || io->n_micro < 0) return fail(XPIPE_EINVAL, "inputs and outputs required");
  xpipe_status s = check_hp(hp);
  if (s != XPIPE_OK) return s;
  if (rule) {
    s = check_rule(rule);
    if (s != XPIPE_OK) return s;
  }
  if (st->has_loss && !io->labels) return fail(XPIPE_EINVAL, "labels required for a loss stage");
  if (!st->has_loss && !io->dy) return fail(XPIPE_EINVAL, "dy required for a stage without a loss");
  // every event is checked before the first launch
  for (int32_t q = 0; q < n_events; ++q) {
    const xpipe_sched_event& e = events[q];
    if (e.micro < 1 || e.micro > io->n_micro || (e.kind != XPIPE_FWD && e.kind != XPIPE_BWD) ||
        (e.bellwether && e.s_eq < 0))
      return fail(XPIPE_EINVAL, "event " + std::to_string(q) + " out of range");
  }
  xpipe_hparams h = *hp;
  int64_t bell_t = -1, cache_t = -1;  // update counts at the forward bellwether / cached forward prediction
  int32_t bell_s = 0;
  for (int32_t q = 0; q < n_events; ++q) {
    const xpipe_sched_event& e = events[q];
    const int32_t k = e.micro - 1;
    if (e.kind == XPIPE_FWD) {
      if (e.bellwether) {
        s = xpipe_predict_weights(st, XPIPE_FWD, e.s_eq, &h);
        bell_s = e.s_eq;
        bell_t = cache_t = h.t;
      } else if (draft && bell_t >= 0 && cache_t != h.t) {
        const int64_t left = (int64_t)bell_s - (h.t - bell_t);
        s = xpipe_predict_weights(st, XPIPE_FWD, (int32_t)(left > 0 ? left : 0), &h);
        cache_t = h.t;
      }
      if (s != XPIPE_OK) return s;
      s = xpipe_stage_fwd(st, io->x[k], io->y[k], io->labels ? io->labels[k] : nullptr,
                          io->loss ? io->loss + k : nullptr);
    } else {
      if (e.bellwether) {
        s = xpipe_predict_weights(st, XPIPE_BWD, e.s_eq, &h);
        if (s != XPIPE_OK) return s;
      }
      s = xpipe_stage_bwd(st, io->x[k], io->dy ? io->dy[k] : nullptr, io->labels ? io->labels[k] : nullptr,
                          io->dx ? io->dx[k] : nullptr);
      if (s == XPIPE_OK && e.update_after) {
        s = rule ? xpipe_rule_step(st, rule, &h, buf, sq, 0, 0, XPIPE_KEEP_PRED)
                 : xpipe_adam_step(st, &h, 0, 0, XPIPE_KEEP_PRED);
        ++h.t;
      }
    }
    if (s != XPIPE_OK) return s;
  }
  return XPIPE_OK;
}

// ============================================================================
// Model partition (Sec. IV-B)
// ============================================================================
xpipe_status xpipe_partition(const xpipe_layer_desc* layers, int32_t n_layers, int32_t stages, int32_t* first) {
  if (!layers || !first || n_layers <= 0 || stages < 1) return fail(XPIPE_EINVAL, "bad arguments");
  std::vector<int32_t> wl;
  for (int32_t i = 0; i < n_layers; ++i) {
    const xpipe_layer_desc& d = layers[i];
    if (d.n_inputs < 1 || d.n_inputs > XPIPE_MAX_INPUTS) return fail(XPIPE_EINVAL, "bad input count");
    for (int32_t q = 0; q < d.n_inputs; ++q)
      if (d.inputs[q] >= i || d.inputs[q] < -1) return fail(XPIPE_EINVAL, "layer inputs must precede the layer");
    if (d.kind == XPIPE_LINEAR || d.kind == XPIPE_CONV) wl.push_back(i);
  }
  const int32_t L = (int32_t)wl.size();
  if (stages > L) return fail(XPIPE_EINVAL, "more stages than layers with weights");
  // a cut before layer c is valid when every layer from c on reads nothing
  // older than layer c - 1 (the hand-off): suffix minimum of the inputs
  std::vector<int32_t> sm(n_layers + 1, n_layers);
  for (int32_t i = n_layers - 1; i >= 0; --i) {
    int32_t m = sm[i + 1];
    for (int32_t q = 0; q < layers[i].n_inputs; ++q) m = std::min(m, layers[i].inputs[q]);
    sm[i] = m;
  }
  auto valid = [&](int32_t j) { return sm[wl[j]] >= wl[j] - 1; };
  // stage k takes L / K weighted layers, the last L % K stages one more; a cut
  // that would split a branch or a skip connection moves to the nearest valid
  // cut (ties: the earlier one, so the later stage takes the extra layers)
  const int32_t base = L / stages, rem = L % stages;
  first[0] = 0;
  int32_t target = 0, prev = 0;
  for (int32_t k = 1; k < stages; ++k) {
    target += base + (k - 1 >= stages - rem ? 1 : 0);
    const int32_t hi = L - (stages - k);  // leave a weighted layer for every later stage
    int32_t best = -1;
    for (int32_t j = prev + 1; j <= hi; ++j)
      if (valid(j) && (best < 0 || std::abs(j - target) < std::abs(best - target))) best = j;
    if (best < 0)
      return fail(XPIPE_EUNSUPPORTED, "no valid cut for stage " + std::to_string(k) +
                                          ": every cut in range splits a branch or a skip connection");
    first[k] = wl[best];
    prev = best;
  }
  first[stages] = n_layers;
  // every layer reads only its own stage, or the previous stage's last layer
  for (int32_t k = 0; k < stages; ++k)
    for (int32_t i = first[k]; i < first[k + 1]; ++i)
      for (int32_t q = 0; q < layers[i].n_inputs; ++q) {
        const int32_t j = layers[i].inputs[q];
        if (j >= first[k] || (k == 0 ? j == -1 : j == first[k] - 1)) continue;
        return fail(XPIPE_EUNSUPPORTED, "layer " + std::to_string(i) + " of stage " + std::to_string(k) +
                                            " reads layer " + std::to_string(j) + " across a stage boundary");
      }
  return XPIPE_OK;
}
