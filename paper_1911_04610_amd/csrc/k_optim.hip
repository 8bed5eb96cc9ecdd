// Weight prediction (Eq. 3) and the Adam update (Eq. 4 moments, Kingma-Ba
// step) over flat fp32 buffers: bandwidth-bound streaming kernels.
//
// Each thread moves 16-byte vectors (global_load_dwordx4) with non-temporal
// hints (the buffers are read once per call and far exceed the caches at
// production sizes); no LDS.  Arithmetic is done in fp64 and rounded once to
// fp32 on store, so a stored value is the nearest fp32 of the exact formula
// evaluated on the stored inputs.
#include "xp_device.h"
#include "xp_kernels.h"

namespace xp {

thread_local LaunchHook* g_hook = nullptr;

// threads per workgroup of the streaming passes (prediction, updates)
constexpr int STREAM_BLOCK = 256;

XP_DEV double pred_dir(double m, double v, const PredCoef& c) {
  double mh = m * c.c1, vh = v * c.c2;
  if (c.kind == PRED_DIR_SMOOTHED) return mh;
  return c.kind == PRED_DIR_ADAM ? mh / (sqrt(vh) + c.eps) : mh / sqrt(vh + c.eps);
}

// s = 0 (or t = 0 with bias correction) is the identity: W is returned bit for bit
XP_DEV float predict1(float w, float m, float v, const PredCoef& c) {
  if (c.coef == 0.0) return w;
  return (float)((double)w - c.coef * pred_dir((double)m, (double)v, c));
}

// both predictions of the fused update: one direction when the two
// coefficient sets share it (same moments' scales and eps, s differs), the
// same fp64 operations as two separate predict1 calls
XP_DEV void predict2(float w, float m, float v, const PredCoef& cf, const PredCoef& cb, bool shared,
                     float& rf, float& rb) {
  if (!shared) {
    rf = predict1(w, m, v, cf);
    rb = predict1(w, m, v, cb);
    return;
  }
  const double d = (cf.coef == 0.0 && cb.coef == 0.0) ? 0.0 : pred_dir((double)m, (double)v, cf);
  rf = cf.coef == 0.0 ? w : (float)((double)w - cf.coef * d);
  rb = cb.coef == 0.0 ? w : (float)((double)w - cb.coef * d);
}

typedef float nf4 __attribute__((ext_vector_type(4)));
typedef uint32_t nu2 __attribute__((ext_vector_type(2)));

// streaming (non-temporal) 16-byte / 8-byte accesses
XP_DEV float4 ldnt(const float4* p) {
  nf4 v = __builtin_nontemporal_load(reinterpret_cast<const nf4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
XP_DEV void stnt(float4* p, float4 v) {
  nf4 r = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(r, reinterpret_cast<nf4*>(p));
}
XP_DEV void stnt(uint2* p, uint2 v) {
  nu2 r = {v.x, v.y};
  __builtin_nontemporal_store(r, reinterpret_cast<nu2*>(p));
}

// ---------------------------------------------------------------- predict
__global__ __launch_bounds__(STREAM_BLOCK) void k_predict(const float* __restrict__ W,
                                                  const float* __restrict__ m,
                                                  const float* __restrict__ v,
                                                  float* __restrict__ out,
                                                  bf16_t* __restrict__ out_bf, int64_t n,
                                                  PredCoef c) {
  const int64_t nv = n >> 2;  // float4 chunks (buffers are 16-byte aligned)
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float4* W4 = reinterpret_cast<const float4*>(W);
  const float4* m4 = reinterpret_cast<const float4*>(m);
  const float4* v4 = reinterpret_cast<const float4*>(v);
  float4* o4 = reinterpret_cast<float4*>(out);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    float4 w = ldnt(W4 + i), mm = ldnt(m4 + i), vv = ldnt(v4 + i);
    float4 r;
    r.x = predict1(w.x, mm.x, vv.x, c);
    r.y = predict1(w.y, mm.y, vv.y, c);
    r.z = predict1(w.z, mm.z, vv.z, c);
    r.w = predict1(w.w, mm.w, vv.w, c);
    stnt(o4 + i, r);
    if (out_bf) {
      uint2 b;
      b.x = f32x2_to_bf16x2(r.x, r.y);
      b.y = f32x2_to_bf16x2(r.z, r.w);
      stnt(reinterpret_cast<uint2*>(out_bf) + i, b);
    }
  }
  // scalar tail
  int64_t t = (nv << 2) + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) {
    float r = predict1(W[t], m[t], v[t], c);
    out[t] = r;
    if (out_bf) out_bf[t] = f32_to_bf16(r);
  }
}

// ---------------------------------------------------------------- adam (+zero grad, +predictions)
struct AdamElem {
  float w, m, v;
};

// The moment recurrences are evaluated operation by operation (no fused
// multiply-add) in the order beta*m + ((1-beta)*g) and beta*v + (((1-beta)*g)*g):
// for fp32 inputs the exact result often falls exactly halfway between two
// fp32 values, and only an identical sequence of roundings settles such ties
// the same way as a reference evaluated in that order.
XP_DEV AdamElem adam1(float w, float m, float v, float g, const AdamCoef& a) {
#pragma clang fp contract(off)
  double gd = (double)g;
  double mn = a.beta1 * (double)m + a.one_m_beta1 * gd;
  double vn = a.beta2 * (double)v + (a.one_m_beta2 * gd) * gd;
  double wn = (double)w - a.lr * (mn * a.bc1) / (sqrt(vn * a.bc2) + a.eps);
  return AdamElem{(float)wn, (float)mn, (float)vn};
}

__global__ __launch_bounds__(STREAM_BLOCK) void k_adam(float* __restrict__ W, float* __restrict__ m,
                                               float* __restrict__ v, float* __restrict__ G,
                                               int64_t n, AdamCoef a, int zero_grad,
                                               float* __restrict__ pf, bf16_t* __restrict__ pf_bf,
                                               PredCoef cf, float* __restrict__ pb,
                                               bf16_t* __restrict__ pb_bf, PredCoef cb) {
  const int64_t nv = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const bool shared = cf.c1 == cb.c1 && cf.c2 == cb.c2 && cf.eps == cb.eps && cf.kind == cb.kind;
  float4* W4 = reinterpret_cast<float4*>(W);
  float4* m4 = reinterpret_cast<float4*>(m);
  float4* v4 = reinterpret_cast<float4*>(v);
  float4* G4 = reinterpret_cast<float4*>(G);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    float4 w = ldnt(W4 + i), mm = ldnt(m4 + i), vv = ldnt(v4 + i), g = ldnt(G4 + i);
    AdamElem e0 = adam1(w.x, mm.x, vv.x, g.x, a);
    AdamElem e1 = adam1(w.y, mm.y, vv.y, g.y, a);
    AdamElem e2 = adam1(w.z, mm.z, vv.z, g.z, a);
    AdamElem e3 = adam1(w.w, mm.w, vv.w, g.w, a);
    stnt(W4 + i, make_float4(e0.w, e1.w, e2.w, e3.w));
    stnt(m4 + i, make_float4(e0.m, e1.m, e2.m, e3.m));
    stnt(v4 + i, make_float4(e0.v, e1.v, e2.v, e3.v));
    if (zero_grad) stnt(G4 + i, make_float4(0.f, 0.f, 0.f, 0.f));
    if (pf && pb) {
      float4 rf, rb;
      predict2(e0.w, e0.m, e0.v, cf, cb, shared, rf.x, rb.x);
      predict2(e1.w, e1.m, e1.v, cf, cb, shared, rf.y, rb.y);
      predict2(e2.w, e2.m, e2.v, cf, cb, shared, rf.z, rb.z);
      predict2(e3.w, e3.m, e3.v, cf, cb, shared, rf.w, rb.w);
      stnt(reinterpret_cast<float4*>(pf) + i, rf);
      stnt(reinterpret_cast<float4*>(pb) + i, rb);
      if (pf_bf) {
        uint2 b;
        b.x = f32x2_to_bf16x2(rf.x, rf.y);
        b.y = f32x2_to_bf16x2(rf.z, rf.w);
        stnt(reinterpret_cast<uint2*>(pf_bf) + i, b);
      }
      if (pb_bf) {
        uint2 b;
        b.x = f32x2_to_bf16x2(rb.x, rb.y);
        b.y = f32x2_to_bf16x2(rb.z, rb.w);
        stnt(reinterpret_cast<uint2*>(pb_bf) + i, b);
      }
    } else if (pf || pb) {
      const PredCoef& c = pf ? cf : cb;
      float* o = pf ? pf : pb;
      bf16_t* ob = pf ? pf_bf : pb_bf;
      float4 r = make_float4(predict1(e0.w, e0.m, e0.v, c), predict1(e1.w, e1.m, e1.v, c),
                             predict1(e2.w, e2.m, e2.v, c), predict1(e3.w, e3.m, e3.v, c));
      stnt(reinterpret_cast<float4*>(o) + i, r);
      if (ob) {
        uint2 b;
        b.x = f32x2_to_bf16x2(r.x, r.y);
        b.y = f32x2_to_bf16x2(r.z, r.w);
        stnt(reinterpret_cast<uint2*>(ob) + i, b);
      }
    }
  }
  int64_t t = (nv << 2) + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) {
    AdamElem e = adam1(W[t], m[t], v[t], G[t], a);
    W[t] = e.w;
    m[t] = e.m;
    v[t] = e.v;
    if (zero_grad) G[t] = 0.f;
    if (pf) {
      float r = predict1(e.w, e.m, e.v, cf);
      pf[t] = r;
      if (pf_bf) pf_bf[t] = f32_to_bf16(r);
    }
    if (pb) {
      float r = predict1(e.w, e.m, e.v, cb);
      pb[t] = r;
      if (pb_bf) pb_bf[t] = f32_to_bf16(r);
    }
  }
}

// ---------------------------------------------------------------- momentum SGD / RMSProp
// The update rules of the paper's other settings, each keeping the Adam
// moments that the prediction reads, all advanced by the same gradient
// g = G + wd * W.  Evaluated in fp64 in the order of the formulas (no fused
// multiply-add), each stored value rounded once to fp32.
struct RuleElem {
  float w, b, q, m, v;  // weight, momentum buffer, squared average, moments
};

template <int RULE>
XP_DEV RuleElem rule1(float w, float b, float q, float m, float v, float gr, const RuleCoef& c) {
#pragma clang fp contract(off)
  const double wd = (double)w;
  const double g = (double)gr + c.wd * wd;
  double qn = 0.0, bn;
  if constexpr (RULE == RULE_MOMENTUM_SGD) {
    bn = c.mu * (double)b + g;
  } else {
    qn = c.alpha * (double)q + (c.one_m_alpha * g) * g;
    bn = c.mu * (double)b + g / (sqrt(qn) + c.eps);
  }
  const double wn = wd - c.lr * bn;
  const double mn = c.beta1 * (double)m + c.one_m_beta1 * g;
  const double vn = c.beta2 * (double)v + (c.one_m_beta2 * g) * g;
  return RuleElem{(float)wn, (float)bn, (float)qn, (float)mn, (float)vn};
}

template <int RULE>
__global__ __launch_bounds__(STREAM_BLOCK) void k_rule(float* __restrict__ W, float* __restrict__ B,
                                              float* __restrict__ Q, float* __restrict__ m,
                                              float* __restrict__ v, float* __restrict__ G, int64_t n,
                                              RuleCoef c, int zero_grad, float* __restrict__ pf,
                                              bf16_t* __restrict__ pf_bf, PredCoef cf,
                                              float* __restrict__ pb, bf16_t* __restrict__ pb_bf,
                                              PredCoef cb) {
  constexpr bool RMS = RULE == RULE_RMSPROP;
  const int64_t nv = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  float4* W4 = reinterpret_cast<float4*>(W);
  float4* B4 = reinterpret_cast<float4*>(B);
  float4* Q4 = reinterpret_cast<float4*>(Q);
  float4* m4 = reinterpret_cast<float4*>(m);
  float4* v4 = reinterpret_cast<float4*>(v);
  float4* G4 = reinterpret_cast<float4*>(G);
  const bool shared = cf.c1 == cb.c1 && cf.c2 == cb.c2 && cf.eps == cb.eps && cf.kind == cb.kind;
  auto preds = [&](int64_t i, const RuleElem (&e)[4]) __attribute__((always_inline)) {
    if (pf && pb) {
      float4 rf, rb;
      predict2(e[0].w, e[0].m, e[0].v, cf, cb, shared, rf.x, rb.x);
      predict2(e[1].w, e[1].m, e[1].v, cf, cb, shared, rf.y, rb.y);
      predict2(e[2].w, e[2].m, e[2].v, cf, cb, shared, rf.z, rb.z);
      predict2(e[3].w, e[3].m, e[3].v, cf, cb, shared, rf.w, rb.w);
      stnt(reinterpret_cast<float4*>(pf) + i, rf);
      stnt(reinterpret_cast<float4*>(pb) + i, rb);
      if (pf_bf) stnt(reinterpret_cast<uint2*>(pf_bf) + i,
                      make_uint2(f32x2_to_bf16x2(rf.x, rf.y), f32x2_to_bf16x2(rf.z, rf.w)));
      if (pb_bf) stnt(reinterpret_cast<uint2*>(pb_bf) + i,
                      make_uint2(f32x2_to_bf16x2(rb.x, rb.y), f32x2_to_bf16x2(rb.z, rb.w)));
      return;
    }
    if (pf) {
      float4 r = make_float4(predict1(e[0].w, e[0].m, e[0].v, cf), predict1(e[1].w, e[1].m, e[1].v, cf),
                             predict1(e[2].w, e[2].m, e[2].v, cf), predict1(e[3].w, e[3].m, e[3].v, cf));
      stnt(reinterpret_cast<float4*>(pf) + i, r);
      if (pf_bf) stnt(reinterpret_cast<uint2*>(pf_bf) + i,
                      make_uint2(f32x2_to_bf16x2(r.x, r.y), f32x2_to_bf16x2(r.z, r.w)));
    }
    if (pb) {
      float4 r = make_float4(predict1(e[0].w, e[0].m, e[0].v, cb), predict1(e[1].w, e[1].m, e[1].v, cb),
                             predict1(e[2].w, e[2].m, e[2].v, cb), predict1(e[3].w, e[3].m, e[3].v, cb));
      stnt(reinterpret_cast<float4*>(pb) + i, r);
      if (pb_bf) stnt(reinterpret_cast<uint2*>(pb_bf) + i,
                      make_uint2(f32x2_to_bf16x2(r.x, r.y), f32x2_to_bf16x2(r.z, r.w)));
    }
  };
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
    const float4 w = ldnt(W4 + i), b = ldnt(B4 + i), mm = ldnt(m4 + i), vv = ldnt(v4 + i), g = ldnt(G4 + i);
    const float4 q = RMS ? ldnt(Q4 + i) : make_float4(0.f, 0.f, 0.f, 0.f);
    const RuleElem e[4] = {rule1<RULE>(w.x, b.x, q.x, mm.x, vv.x, g.x, c),
                           rule1<RULE>(w.y, b.y, q.y, mm.y, vv.y, g.y, c),
                           rule1<RULE>(w.z, b.z, q.z, mm.z, vv.z, g.z, c),
                           rule1<RULE>(w.w, b.w, q.w, mm.w, vv.w, g.w, c)};
    stnt(W4 + i, make_float4(e[0].w, e[1].w, e[2].w, e[3].w));
    stnt(B4 + i, make_float4(e[0].b, e[1].b, e[2].b, e[3].b));
    if (RMS) stnt(Q4 + i, make_float4(e[0].q, e[1].q, e[2].q, e[3].q));
    stnt(m4 + i, make_float4(e[0].m, e[1].m, e[2].m, e[3].m));
    stnt(v4 + i, make_float4(e[0].v, e[1].v, e[2].v, e[3].v));
    if (zero_grad) stnt(G4 + i, make_float4(0.f, 0.f, 0.f, 0.f));
    preds(i, e);
  }
  const int64_t t = (nv << 2) + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < n) {
    const RuleElem e = rule1<RULE>(W[t], B[t], RMS ? Q[t] : 0.f, m[t], v[t], G[t], c);
    W[t] = e.w;
    B[t] = e.b;
    if (RMS) Q[t] = e.q;
    m[t] = e.m;
    v[t] = e.v;
    if (zero_grad) G[t] = 0.f;
    if (pf) {
      const float r = predict1(e.w, e.m, e.v, cf);
      pf[t] = r;
      if (pf_bf) pf_bf[t] = f32_to_bf16(r);
    }
    if (pb) {
      const float r = predict1(e.w, e.m, e.v, cb);
      pb[t] = r;
      if (pb_bf) pb_bf[t] = f32_to_bf16(r);
    }
  }
}

// ---------------------------------------------------------------- launchers
static int stream_grid(int64_t n) {
  // one 16-byte vector per thread: every load of the pass is issued up front
  // (measured on MI355X at 1e8 parameters: 6.35 TB/s for the prediction versus
  // 5.3 TB/s with a 2048-workgroup grid-stride loop; 1024-thread workgroups
  // gain ~1.5% on a bare three-read one-write stream but lose more on the
  // passes with fp64 square roots and divides)
  int64_t nv = (n >> 2) + 1;
  int64_t blocks = (nv + STREAM_BLOCK - 1) / STREAM_BLOCK;
  if (blocks > ((int64_t)1 << 30)) blocks = (int64_t)1 << 30;
  if (blocks < 1) blocks = 1;
  return (int)blocks;
}

hipError_t launch_predict(const float* W, const float* m, const float* v, float* out,
                          bf16_t* out_bf, int64_t n, const PredCoef& c, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  XP_LAUNCH("k_predict", (double)n * (out_bf ? 18 : 16), k_predict, dim3(stream_grid(n)), dim3(STREAM_BLOCK), 0, s,
            W, m, v, out, out_bf, n, c);
  return hipGetLastError();
}

hipError_t launch_adam(float* W, float* m, float* v, float* G, int64_t n, const AdamCoef& a,
                       int zero_grad, float* pf, bf16_t* pf_bf, const PredCoef& cf, float* pb,
                       bf16_t* pb_bf, const PredCoef& cb, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  double bytes = (double)n * (28 + (zero_grad ? 4 : 0) + (pf ? 4 : 0) + (pb ? 4 : 0) +
                              (pf_bf ? 2 : 0) + (pb_bf ? 2 : 0));
  XP_LAUNCH("k_adam", bytes, k_adam, dim3(stream_grid(n)), dim3(STREAM_BLOCK), 0, s, W, m, v, G, n, a, zero_grad,
            pf, pf_bf, cf, pb, pb_bf, cb);
  return hipGetLastError();
}

hipError_t launch_rule(int rule, float* W, float* B, float* Q, float* m, float* v, float* G, int64_t n,
                       const RuleCoef& c, int zero_grad, float* pf, bf16_t* pf_bf, const PredCoef& cf,
                       float* pb, bf16_t* pb_bf, const PredCoef& cb, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool rms = rule == RULE_RMSPROP;
  double bytes = (double)n * ((rms ? 44 : 36) + (zero_grad ? 4 : 0) + (pf ? 4 : 0) + (pb ? 4 : 0) +
                              (pf_bf ? 2 : 0) + (pb_bf ? 2 : 0));
  if (rms)
    XP_LAUNCH("k_rule<rmsprop>", bytes, k_rule<RULE_RMSPROP>, dim3(stream_grid(n)), dim3(STREAM_BLOCK), 0, s, W, B, Q,
              m, v, G, n, c, zero_grad, pf, pf_bf, cf, pb, pb_bf, cb);
  else
    XP_LAUNCH("k_rule<momentum_sgd>", bytes, k_rule<RULE_MOMENTUM_SGD>, dim3(stream_grid(n)), dim3(STREAM_BLOCK), 0, s,
              W, B, Q, m, v, G, n, c, zero_grad, pf, pf_bf, cf, pb, pb_bf, cb);
  return hipGetLastError();
}

// ---------------------------------------------------------------- measurement probes
__global__ __launch_bounds__(256) void k_probe_copy(const uint4* __restrict__ src,
                                                     uint4* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_probe_mfma(float* out, int waves, int iters) {
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(float)((lane + e) & 7);
    b[e] = (__bf16)(float)((lane * 3 + e) & 7);
  }
  f32x16_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[j][r];
  if (lane == 0 && wave < waves) out[wave] = s;
}

hipError_t launch_probe_copy(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  const int64_t n = bytes / 16;
  if (n <= 0) return hipSuccess;
  XP_LAUNCH("k_probe_copy", (double)bytes * 2, k_probe_copy, dim3((unsigned)((n + 255) / 256)),
            dim3(256), 0, s, (const uint4*)src, (uint4*)dst, n);
  return hipGetLastError();
}

// a bare stream of the passes' shape: nsrc 16-byte reads and ndst 16-byte
// writes per thread (non-temporal, as the passes), one add per element
__global__ __launch_bounds__(256) void k_probe_stream(StreamArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < STREAM_MAX_SRC; ++j)
    if (j < a.nsrc) {
      const float4 v = ldnt(reinterpret_cast<const float4*>(a.src[j]) + i);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
#pragma unroll
  for (int j = 0; j < STREAM_MAX_DST; ++j)
    if (j < a.ndst) stnt(reinterpret_cast<float4*>(a.dst[j]) + i, acc);
}

hipError_t launch_probe_stream(const StreamArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  XP_LAUNCH("k_probe_stream", (double)a.n * 16 * (a.nsrc + a.ndst), k_probe_stream,
            dim3((unsigned)((a.n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// graph probe: a fixed amount of dependent fp32 work per thread (iters
// multiply-adds on one value), one float written per launch so it is kept
__global__ __launch_bounds__(256) void k_probe_spin(float* p, int i, int iters) {
  float v = p[i & 1023];
  for (int k = 0; k < iters; ++k) v = v * 0.999f + 1.0f;
  if (threadIdx.x == 0 && blockIdx.x == 0) p[1024 + (i & 1023)] = v;
}

hipError_t launch_probe_spin(float* p, int i, int iters, int blocks, hipStream_t s) {
  XP_LAUNCH("k_probe_spin", 0.0, k_probe_spin, dim3(blocks), dim3(256), 0, s, p, i, iters);
  return hipGetLastError();
}

hipError_t launch_probe_mfma(float* out, int waves, int iters, hipStream_t s) {
  if (waves <= 0 || iters <= 0) return hipSuccess;
  XP_LAUNCH("k_probe_mfma", (double)waves * iters * 8 * 32768.0, k_probe_mfma,
            dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, out, waves, iters);
  return hipGetLastError();
}

}  // namespace xp
