// Host side of libfeatfix.so: argument validation, the fixed schedule (plan), the
// exact-block composer, the per-step executor and the C ABI of include/featfix.h.
// The library owns host objects only; every device buffer is the caller's.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "featfix.h"
#include "kernels.h"

using namespace ff;

namespace ff {
thread_local LaunchEvents g_launch_events;
}

namespace {

thread_local char g_err[512] = "";

ff_status fail(ff_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}
ff_status ok() {
  g_err[0] = 0;
  return FF_OK;
}
ff_status hip_fail(hipError_t e, const char* where) {
  return fail(FF_E_HIP, "%s: %s", where, hipGetErrorString(e));
}
#define HIP_TRY(expr, where)              \
  do {                                    \
    hipError_t _e = (expr);               \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---------------------------------------------------------------- model validation
struct Model {
  int L = 0;
  std::vector<int> kinds;
  int C = 0, H = 0, d = 0, M = 0, n_img = 0, n_txt = 0, B = 0, N = 0, P = 0;
  int lat_c = 0, lat_f = 0, lat_h = 0, lat_w = 0, pt = 0, ph = 0, pw = 0;
  int dtype = 0;
  float ln_eps = 0.f;
  int rope[3] = {0, 0, 0};
  float rope_theta = 0.f;
  int cfg = 0;            // classifier-free guidance pairs (rows b, b + B/2)
  float cfg_scale = 0.f;
  bool any_single = false;
  size_t es() const { return dsize(dtype); }
  size_t E() const { return (size_t)B * N * C; }
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// the rotary embedding of the q / k norm kernel (axes 0: none)
Rope rope_of(const Model& m) {
  Rope r{};
  for (int a = 0; a < 3; ++a) r.axes[a] = m.rope[a];
  r.log2_theta = m.rope[0] + m.rope[1] + m.rope[2] ? log2f(m.rope_theta) : 0.f;
  r.n_txt = m.n_txt;
  r.Hp = m.lat_h / m.ph;
  r.Wp = m.lat_w / m.pw;
  return r;
}

ff_status check_model(const ff_model_desc* m, Model* out) {
  if (!m) return fail(FF_E_NULL, "model descriptor is NULL");
  if (m->dtype != FF_F32 && m->dtype != FF_BF16) return fail(FF_E_DTYPE, "unknown dtype %d", m->dtype);
  if (m->n_layers < 1 || m->n_layers > 4096) return fail(FF_E_SHAPE, "n_layers %d out of range", m->n_layers);
  if (!m->kinds) return fail(FF_E_NULL, "kinds is NULL");
  Model r;
  r.L = m->n_layers;
  r.C = m->C; r.H = m->H; r.d = m->d; r.M = m->mlp_hidden;
  r.n_img = m->n_img; r.n_txt = m->n_txt; r.B = m->B;
  r.lat_c = m->lat_c; r.lat_f = m->lat_f; r.lat_h = m->lat_h; r.lat_w = m->lat_w;
  r.pt = m->pt; r.ph = m->ph; r.pw = m->pw;
  r.dtype = m->dtype;
  r.ln_eps = m->ln_eps;
  for (int l = 0; l < r.L; ++l) {
    const int k = m->kinds[l];
    if (k != FF_DIT && k != FF_MMDIT_DOUBLE && k != FF_MMDIT_SINGLE)
      return fail(FF_E_SHAPE, "layer %d: unknown block kind %d", l, k);
    if (k == FF_DIT && r.n_txt != 0) return fail(FF_E_SHAPE, "layer %d: DiT blocks need n_txt == 0", l);
    if (k == FF_MMDIT_SINGLE) r.any_single = true;
    r.kinds.push_back(k);
  }
  if (r.B < 1 || r.B > kGemvMaxB) return fail(FF_E_SHAPE, "batch %d outside [1, %d]", r.B, kGemvMaxB);
  if (r.H < 1 || r.d < 8 || r.d > 128 || r.d % 8 || (long)r.H * r.d != r.C)
    return fail(FF_E_SHAPE, "need C == H*d, 8 <= d <= 128, d %% 8 == 0 (C=%d H=%d d=%d)", r.C, r.H, r.d);
  const int cmax = r.dtype == FF_BF16 ? 4096 : 2048;
  if (r.C % 8 || r.C > cmax) return fail(FF_E_SHAPE, "C=%d must be a multiple of 8 and <= %d", r.C, cmax);
  if (r.M < 8 || r.M % 8) return fail(FF_E_SHAPE, "mlp_hidden=%d must be a positive multiple of 8", r.M);
  if (r.n_img < 1 || r.n_txt < 0) return fail(FF_E_SHAPE, "bad token counts n_img=%d n_txt=%d", r.n_img, r.n_txt);
  if (r.pt < 1 || r.ph < 1 || r.pw < 1 || r.lat_c < 1 || r.lat_f < 1 || r.lat_h < 1 || r.lat_w < 1)
    return fail(FF_E_SHAPE, "bad latent / patch geometry");
  if (r.lat_f % r.pt || r.lat_h % r.ph || r.lat_w % r.pw) return fail(FF_E_SHAPE, "latent not divisible by patch");
  const long nimg = (long)(r.lat_f / r.pt) * (r.lat_h / r.ph) * (r.lat_w / r.pw);
  if (nimg != r.n_img) return fail(FF_E_SHAPE, "n_img=%d but the latent has %ld patches", r.n_img, nimg);
  r.P = r.pt * r.ph * r.pw * r.lat_c;
  if (r.P % 8) return fail(FF_E_SHAPE, "patch features %d must be a multiple of 8", r.P);
  const int rsum = m->rope_axes[0] + m->rope_axes[1] + m->rope_axes[2];
  if (rsum != 0) {
    for (int a = 0; a < 3; ++a)
      if (m->rope_axes[a] < 0 || m->rope_axes[a] % 2) return fail(FF_E_SHAPE, "rope_axes must be even and >= 0");
    if (rsum != r.d) return fail(FF_E_SHAPE, "rope_axes sum to %d, head dim is %d", rsum, r.d);
    if (!(m->rope_theta > 1.f) || !std::isfinite(m->rope_theta)) return fail(FF_E_RANGE, "rope_theta must be > 1");
    for (int a = 0; a < 3; ++a) r.rope[a] = m->rope_axes[a];
    r.rope_theta = m->rope_theta;
  }
  if (m->cfg_pairs != 0 && m->cfg_pairs != 1) return fail(FF_E_RANGE, "cfg_pairs must be 0 or 1");
  if (m->cfg_pairs) {
    if (r.B % 2) return fail(FF_E_SHAPE, "guidance pairs need an even batch (B=%d)", r.B);
    if (!std::isfinite(m->cfg_scale)) return fail(FF_E_RANGE, "cfg_scale must be finite");
    r.cfg = 1;
    r.cfg_scale = m->cfg_scale;
  }
  r.N = r.n_img + r.n_txt;
  if ((long)r.B * r.N > (1L << 30) / 8) return fail(FF_E_SHAPE, "too many rows");
  if (!(r.ln_eps > 0.f)) return fail(FF_E_RANGE, "ln_eps must be > 0");
  *out = r;
  return FF_OK;
}

// ---------------------------------------------------------------- workspace layout
struct Ws {
  size_t X0, X1, HF, LNA, QKV, ATT, X1F, HID, MOD, CT, CS, TMP, PHI, PATCH, YF, PART, MODS, XS, REL, total;
  size_t mod_slot;   // floats per layer slot of MODS
};

// Modulation vectors per layer kind: 6C (DiT), 2 x 6C (MMDiT double), 3C (MMDiT single).
int mod_floats(int kind, int C) { return kind == FF_MMDIT_DOUBLE ? 12 * C : kind == FF_MMDIT_SINGLE ? 3 * C : 6 * C; }
int mod_width(const Model& m) {
  int w = 0;
  for (int k : m.kinds) w = std::max(w, mod_floats(k, m.C));
  return w;
}
constexpr int kModLayers = kGemvJobs / 2;   // layers whose modulation one batched launch computes

Ws ws_layout(const Model& m) {
  Ws w{};
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  const size_t es = m.es(), rows = (size_t)m.B * m.N;
  w.X0 = take(rows * m.C * es);
  w.X1 = take(rows * m.C * es);
  w.HF = take(rows * m.C * es);
  w.LNA = take(rows * m.C * es);
  w.QKV = take(rows * 3 * (size_t)m.C * es);
  w.ATT = take(rows * (size_t)(m.any_single ? m.C + m.M : m.C) * es);
  w.X1F = take(rows * m.C * 4);
  w.HID = take(rows * (size_t)m.M * es);
  w.MOD = take((size_t)m.B * 12 * m.C * 4);
  w.CT = take((size_t)m.B * m.C * 4);
  w.CS = take((size_t)m.B * m.C * 4);
  w.TMP = take((size_t)m.B * m.C * 4);
  w.PHI = take(FF_TEMB_DIM * 4);
  w.PATCH = take((size_t)m.B * m.n_img * m.P * es);
  w.YF = take((size_t)m.B * m.n_img * m.P * 4);
  w.PART = take(verify_partials_floats(m.B) * 4);
  w.mod_slot = (size_t)m.B * mod_width(m);
  w.MODS = take(kModLayers * w.mod_slot * 4);
  w.XS = take(gemv_xs_bytes(m.C));
  w.REL = take((size_t)m.L * m.B * 4);   // one step's site discrepancies (adaptive refresh)
  w.total = off;
  return w;
}

template <class T = void>
T* at(void* base, size_t off) { return reinterpret_cast<T*>(reinterpret_cast<char*>(base) + off); }


// ---------------------------------------------------------------- launches (+ optional profiling)
// Every kernel launch of the path goes through Exec so that a context with profiling
// enabled can bracket it with HIP events on the same stream and attribute algorithmic
// FLOPs / bytes to its kernel class.
struct Prof {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t next = 0;
  struct Rec { int cls; hipEvent_t a, b; double flops, bytes; };
  std::vector<Rec> recs;
  ~Prof() {
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
  hipError_t get(hipEvent_t* e) {
    if (next == pool.size()) {
      hipEvent_t n;
      hipError_t r = hipEventCreate(&n);
      if (r != hipSuccess) return r;
      pool.push_back(n);
    }
    *e = pool[next++];
    return hipSuccess;
  }
};

struct Exec {
  hipStream_t st;
  Prof* prof;
  int dt;
  size_t es;

  // With profiling on, the launch's (first) kernel is started with a start/stop event pair
  // recorded at its own execution boundaries; a call that launches nothing records nothing.
  template <class F>
  hipError_t timed(int cls, double flops, double bytes, F&& launch) {
    if (!prof || !prof->on) return launch();
    hipEvent_t a, b;
    hipError_t e = prof->get(&a);
    if (e == hipSuccess) e = prof->get(&b);
    if (e != hipSuccess) return e;
    g_launch_events = LaunchEvents{a, b};
    e = launch();
    const bool consumed = g_launch_events.start == nullptr;
    g_launch_events = LaunchEvents{};
    if (e != hipSuccess) return e;
    if (consumed) prof->recs.push_back({cls, a, b, flops, bytes});
    else prof->next -= 2;   // hand the unused pair back
    return hipSuccess;
  }
  hipError_t gemm(const GemmArgs& a) {
    const double bytes = ((double)a.M * a.K + (double)a.N * a.K) * es + (double)a.M * a.N * (a.out_f32 ? 4 : es);
    return timed(FF_PROF_GEMM, 2.0 * a.M * a.N * a.K, bytes, [&] { return ff::gemm(dt, a, st); });
  }
  hipError_t gemm2(const GemmArgs& a0, const GemmArgs& a1) {
    auto fl = [](const GemmArgs& a) { return 2.0 * a.M * a.N * a.K; };
    auto by = [&](const GemmArgs& a) {
      return ((double)a.M * a.K + (double)a.N * a.K) * es + (double)a.M * a.N * (a.out_f32 ? 4 : es);
    };
    return timed(FF_PROF_GEMM, fl(a0) + fl(a1), by(a0) + by(a1), [&] { return ff::gemm2(dt, a0, a1, st); });
  }
  hipError_t attention(const AttnArgs& a) {
    const double rows = (double)a.B * a.N;
    return timed(FF_PROF_ATTN, 4.0 * a.B * (double)a.N * a.N * a.H * a.d, rows * 4.0 * a.C * es,
                 [&] { return ff::attention(dt, a, st); });
  }
  hipError_t gemv_batch(const GemvBatch& b) {
    double fl = 0, by = 0;
    for (int i = 0; i < b.njobs; ++i) {
      fl += 2.0 * b.B * b.job[i].Nout * b.K;
      by += (double)b.job[i].Nout * b.K * es;
    }
    return timed(FF_PROF_GEMV, fl, by, [&] { return ff::gemv_batch(dt, b, st); });
  }
  // a modulation GEMM of the conditioning cache (counted with the GEMVs it replaces)
  hipError_t mod_gemm(const GemmArgs& a) {
    const double bytes = ((double)a.M * a.K + (double)a.N * a.K) * es + (double)a.M * a.N * (a.out_f32 ? 4 : es);
    return timed(FF_PROF_GEMV, 2.0 * a.M * a.N * a.K, bytes, [&] { return ff::gemm(dt, a, st); });
  }
  hipError_t gemv(const GemvArgs& a) {
    return timed(FF_PROF_GEMV, 2.0 * a.B * a.Nout * a.K, (double)a.Nout * a.K * es, [&] { return ff::gemv(dt, a, st); });
  }
  hipError_t ln(const LnModArgs& a) {
    // with a run draft in front (pre.n > 0) the launch also moves the draft's bytes: the
    // history sums read and the updated stream written back; it is counted as a draft
    const double pre = a.pre.n ? 4.0 * a.pre.n + es : 0.0;
    return timed(a.pre.n ? FF_PROF_DRAFT : FF_PROF_NORM, 0, (double)a.rows * a.C * ((a.in_f32 ? 4 : es) + es + pre),
                 [&] { return ff::ln_modulate(dt, a, st); });
  }
  hipError_t rms_qk(const RmsQKArgs& a) {
    return timed(FF_PROF_NORM, 0, 4.0 * a.rows * a.H * a.d * es, [&] { return ff::rms_qk(dt, a, st); });
  }
  hipError_t cache(void* slot, const void* u, const void* h, size_t E) {
    return timed(FF_PROF_CACHE, 0, (u ? 3.0 : 2.0) * E * es, [&] { return ff::cache_update(dt, slot, u, h, E, st); });
  }
  hipError_t draft_run(const Terms& t, int layers, size_t layer_stride, bool resid, void* x, size_t E) {
    return timed(FF_PROF_DRAFT, 0, ((double)t.n * layers + (resid ? 2.0 : 1.0)) * E * es,
                 [&] { return ff::draft_run(dt, t, layers, layer_stride, resid ? 1 : 0, x, E, st); });
  }
  hipError_t hist_sum(const void* slot0, int layers, size_t layer_stride, float* out, size_t E) {
    return timed(FF_PROF_CACHE, 0, ((double)layers * es + 4.0) * E,
                 [&] { return ff::hist_sum(dt, slot0, layers, layer_stride, out, E, st); });
  }
  hipError_t draft_sum(const Terms& t, void* x, size_t E) {
    return timed(FF_PROF_DRAFT, 0, (4.0 * t.n + 2.0 * es) * E, [&] { return ff::draft_sum(dt, t, x, E, st); });
  }
  hipError_t draft(const Terms& t, const void* u, void* hd, size_t E) {
    return timed(FF_PROF_DRAFT, 0, (t.n + (u ? 2.0 : 1.0)) * E * es, [&] { return ff::draft(dt, t, u, hd, E, st); });
  }
  hipError_t verify(const Terms& t, const void* u, const void* hf, void* hout, const Forward& fwd, int B, size_t Eb,
                    float eps, float* rel, float* part) {
    return timed(FF_PROF_VERIFY, 0, (t.n + (u ? 3.0 : 2.0)) * Eb * B * es,
                 [&] { return ff::verify(dt, t, u, hf, hout, fwd, B, Eb, eps, rel, part, st); });
  }
  template <class F>
  hipError_t other(double bytes, F&& launch) { return timed(FF_PROF_OTHER, 0, bytes, launch); }
};

// ---------------------------------------------------------------- weights
bool stream_ok(const ff_stream_weights& s, int kind) {
  if (!s.mod_w || !s.mod_b || !aligned16(s.mod_w)) return false;
  if (kind == FF_MMDIT_SINGLE) {
    if (!s.lin1_w || !s.lin1_b || !s.lin2_w || !s.lin2_b) return false;
    if (!aligned16(s.lin1_w) || !aligned16(s.lin2_w)) return false;
  } else {
    if (!s.qkv_w || !s.qkv_b || !s.o_w || !s.o_b || !s.fc1_w || !s.fc1_b || !s.fc2_w || !s.fc2_b) return false;
    if (!aligned16(s.qkv_w) || !aligned16(s.o_w) || !aligned16(s.fc1_w) || !aligned16(s.fc2_w)) return false;
  }
  if (kind != FF_DIT && (!s.q_g || !s.k_g)) return false;
  return true;
}

ff_status check_layer_weights(const ff_layer_weights* w, int kind, int layer) {
  if (!w) return fail(FF_E_NULL, "layer %d: weights are NULL", layer);
  if (!stream_ok(w->s[0], kind) || (kind == FF_MMDIT_DOUBLE && !stream_ok(w->s[1], kind)))
    return fail(FF_E_NULL, "layer %d: a required weight pointer is NULL or not 16-byte aligned", layer);
  return FF_OK;
}

// ---------------------------------------------------------------- exact block (Eq. 1)
RowMap whole(const Model& m) { return RowMap{m.N, m.N, 0}; }

GemmArgs gemm_args(const void* A, int lda, RowMap amap, const void* W, const void* bias, int M, int N, int K,
                   int epi, void* out, int ldo, RowMap omap) {
  GemmArgs g{};
  g.A = A; g.lda = lda; g.amap = amap;
  g.W = W; g.ldw = K;
  g.bias = bias;
  g.M = M; g.N = N; g.K = K;
  g.epi = epi;
  g.out = out; g.ldo = ldo; g.omap = omap; g.out_f32 = 0;
  return g;
}

const void* offset_rows(const void* p, size_t rows, size_t cols, size_t es) {
  return reinterpret_cast<const char*>(p) + rows * cols * es;
}

// h = B_l(u; c_t) with cs = SiLU(c_t) [B, C] fp32 already in the workspace.
// cache_slot (bf16 only): the history refresh of this layer (slot = h - u, or h when
// !cache_resid) is written by the epilogue of the block's last GEMM, from the same rounded
// h that the separate cache kernel would read back.
// pre (bf16 or fp32 stream): a run of drafted layers in front of the block, applied by the
// block's first LayerNorm(s) from its history sums (u is updated in place, every row
// exactly once: all rows, or the text and the image rows of a double block).
ff_status exec_block(const Model& m, int kind, const ff_layer_weights& w, const float* cs, const void* u,
                     void* h, void* ws, Exec& ex, const float* mod_pre = nullptr, void* cache_slot = nullptr,
                     bool cache_resid = true, const Terms* pre = nullptr) {
  const Ws L = ws_layout(m);
  const int C = m.C, Mh = m.M, dt = m.dtype;
  const size_t es = m.es();
  void* lna = at(ws, L.LNA);
  void* qkv = at(ws, L.QKV);
  void* att = at(ws, L.ATT);
  float* x1f = at<float>(ws, L.X1F);
  void* hid = at(ws, L.HID);
  // modulation: precomputed by the caller (batched over the layers of a step) or here
  float* mod = mod_pre ? const_cast<float*>(mod_pre) : at<float>(ws, L.MOD);
  const float scale = 1.0f / sqrtf((float)m.d);

  AttnArgs aa{};
  aa.qkv = qkv; aa.ldq = 3 * C; aa.B = m.B; aa.N = m.N; aa.H = m.H; aa.d = m.d; aa.C = C; aa.scale = scale;

  if (kind == FF_MMDIT_SINGLE) {
    const ff_stream_weights& s = w.s[0];
    const RowMap all = whole(m);
    const int rows = m.B * m.N;
    if (!mod_pre) {
      GemvArgs gv{cs, C, 0, s.mod_w, s.mod_b, 3 * C, C, m.B, mod, 3 * C, 0, nullptr, 0};
      HIP_TRY(ex.gemv(gv), "single: modulation");
    }
    LnModArgs ln{u, 0, C, all, rows, C, m.ln_eps, mod, mod + C, 3 * C, lna, C};
    if (pre) ln.pre = *pre;
    HIP_TRY(ex.ln(ln), "single: ln");
    // lin1 = [qkv | MLP] over the same input: the two parts (bias, bias + GELU) in one launch
    GemmArgs g1 = gemm_args(lna, C, all, s.lin1_w, s.lin1_b, rows, 3 * C, C, EPI_BIAS, qkv, 3 * C, all);
    const int ldy = C + Mh;
    GemmArgs g2 = gemm_args(lna, C, all, offset_rows(s.lin1_w, 3 * (size_t)C, C, es),
                            offset_rows(s.lin1_b, 3 * (size_t)C, 1, es), rows, Mh, C, EPI_BIAS_GELU,
                            at(att, (size_t)C * es), ldy, all);
    HIP_TRY(ex.gemm2(g1, g2), "single: lin1");
    RmsQKArgs rn{qkv, 3 * C, all, rows, m.H, m.d, s.q_g, s.k_g, m.ln_eps, rope_of(m)};
    HIP_TRY(ex.rms_qk(rn), "single: q/k norm");
    aa.out = att; aa.ldo = ldy;
    HIP_TRY(ex.attention(aa), "single: attention");
    GemmArgs g3 = gemm_args(att, ldy, all, s.lin2_w, s.lin2_b, rows, C, C + Mh, EPI_GATED, h, C, all);
    g3.resid = u; g3.ldr = C; g3.resid_f32 = 0; g3.gate = mod + 2 * C; g3.ldg = 3 * C;
    g3.cache_out = cache_slot; g3.cache_u = cache_resid ? u : nullptr;
    HIP_TRY(ex.gemm(g3), "single: lin2");
    return FF_OK;
  }

  // DiT block (one stream) or MMDiT double block (text rows, then image rows).  The two
  // streams of a double block write disjoint rows of the shared buffers, so each stage runs
  // for both streams before the next one, and every projection of the two streams (same
  // N, K and epilogue, different weights and rows) is one grouped GEMM launch.
  const int nstreams = kind == FF_MMDIT_DOUBLE ? 2 : 1;
  RowMap maps[2];
  int nseg[2];
  if (kind == FF_MMDIT_DOUBLE) {
    maps[0] = RowMap{m.n_txt > 0 ? m.n_txt : 1, m.N, 0}; nseg[0] = m.n_txt;
    maps[1] = RowMap{m.n_img, m.N, m.n_txt}; nseg[1] = m.n_img;
  } else {
    maps[0] = whole(m); nseg[0] = m.N;
  }
  const int ldm = 6 * C * nstreams;
  // the stream GEMMs of one stage: grouped when both streams have rows
  auto run2 = [&](GemmArgs* g, const char* what) -> ff_status {
    const bool has0 = nstreams > 1 && m.B * nseg[0] > 0, has1 = m.B * nseg[nstreams - 1] > 0;
    if (nstreams > 1 && has0 && has1) {
      HIP_TRY(ex.gemm2(g[0], g[1]), what);
    } else {
      for (int si = 0; si < nstreams; ++si)
        if (m.B * nseg[si] > 0) HIP_TRY(ex.gemm(g[si]), what);
    }
    return FF_OK;
  };
  GemmArgs gs[2];
  for (int si = 0; si < nstreams; ++si) {
    const ff_stream_weights& s = w.s[si];
    const int rows = m.B * nseg[si];
    float* ms = mod + 6 * C * si;
    if (!mod_pre) {
      GemvArgs gv{cs, C, 0, s.mod_w, s.mod_b, 6 * C, C, m.B, ms, ldm, 0, nullptr, 0};
      HIP_TRY(ex.gemv(gv), "block: modulation");
    }
    if (rows == 0) continue;
    LnModArgs ln{u, 0, C, maps[si], rows, C, m.ln_eps, ms, ms + C, ldm, lna, C};
    if (pre) ln.pre = *pre;
    HIP_TRY(ex.ln(ln), "block: ln1");
  }
  for (int si = 0; si < nstreams; ++si)
    gs[si] = gemm_args(lna, C, maps[si], w.s[si].qkv_w, w.s[si].qkv_b, m.B * nseg[si], 3 * C, C, EPI_BIAS, qkv, 3 * C,
                       maps[si]);
  if (ff_status e = run2(gs, "block: qkv")) return e;
  if (kind == FF_MMDIT_DOUBLE) {
    for (int si = 0; si < nstreams; ++si) {
      const int rows = m.B * nseg[si];
      if (rows == 0) continue;
      RmsQKArgs rn{qkv, 3 * C, maps[si], rows, m.H, m.d, w.s[si].q_g, w.s[si].k_g, m.ln_eps, rope_of(m)};
      HIP_TRY(ex.rms_qk(rn), "double: q/k norm");
    }
  }
  aa.out = att; aa.ldo = C;
  HIP_TRY(ex.attention(aa), "block: attention");
  for (int si = 0; si < nstreams; ++si) {
    float* ms = mod + 6 * C * si;
    gs[si] = gemm_args(att, C, maps[si], w.s[si].o_w, w.s[si].o_b, m.B * nseg[si], C, C, EPI_GATED, x1f, C, maps[si]);
    gs[si].out_f32 = 1; gs[si].resid = u; gs[si].ldr = C; gs[si].resid_f32 = 0; gs[si].gate = ms + 2 * C; gs[si].ldg = ldm;
  }
  if (ff_status e = run2(gs, "block: proj")) return e;
  for (int si = 0; si < nstreams; ++si) {
    const int rows = m.B * nseg[si];
    if (rows == 0) continue;
    float* ms = mod + 6 * C * si;
    LnModArgs ln{x1f, 1, C, maps[si], rows, C, m.ln_eps, ms + 3 * C, ms + 4 * C, ldm, lna, C};
    HIP_TRY(ex.ln(ln), "block: ln2");
  }
  for (int si = 0; si < nstreams; ++si)
    gs[si] = gemm_args(lna, C, maps[si], w.s[si].fc1_w, w.s[si].fc1_b, m.B * nseg[si], Mh, C, EPI_BIAS_GELU, hid, Mh,
                       maps[si]);
  if (ff_status e = run2(gs, "block: fc1")) return e;
  for (int si = 0; si < nstreams; ++si) {
    float* ms = mod + 6 * C * si;
    gs[si] = gemm_args(hid, Mh, maps[si], w.s[si].fc2_w, w.s[si].fc2_b, m.B * nseg[si], C, Mh, EPI_GATED, h, C, maps[si]);
    gs[si].resid = x1f; gs[si].ldr = C; gs[si].resid_f32 = 1; gs[si].gate = ms + 5 * C; gs[si].ldg = ldm;
    gs[si].cache_out = cache_slot; gs[si].cache_u = cache_resid ? u : nullptr;
  }
  if (ff_status e = run2(gs, "block: fc2")) return e;
  return FF_OK;
}

// ---------------------------------------------------------------- schedule
}  // namespace

struct ff_plan {
  ff_sched_desc s;
  int L;
  std::vector<int32_t> step_kind, refresh_ord, k_eff, read_slots, write_slot, action;
  std::vector<float> coeffs;
  std::vector<uint8_t> mask;   // [T * L] as given (the adaptive schedule re-reads it)
  ff_counts counts;
};

namespace {

// Coefficients of the Taylor draft in terms of the ring of raw refresh features.
// D^k at refresh j is kept as a combination sum_m W[k][m] * Delta_{j-m}; the recursion
// D^{k+1}_new = (D^k_new - D^k_old) / (tau_j - tau_{j-1}) becomes a recursion on W
// (D^k_old's combination refers to refresh j-1, i.e. is shifted by one ring position).
struct CoefState {
  int K;
  int j = -1;
  double tau = 0;
  double Wk[FF_MAX_K + 1][FF_MAX_K + 2] = {};
  explicit CoefState(int k) : K(k) {}
  void refresh(double tau_new) {
    const int jn = j + 1;
    double nw[FF_MAX_K + 1][FF_MAX_K + 2] = {};
    nw[0][0] = 1.0;
    const int upto = jn < K ? jn : K;
    for (int k = 0; k < upto; ++k) {
      const double gap = tau_new - tau;
      for (int q = 0; q <= K; ++q) {
        const double old_shift = q >= 1 ? Wk[k][q - 1] : 0.0;
        nw[k + 1][q] = (nw[k][q] - old_shift) / gap;
      }
    }
    memcpy(Wk, nw, sizeof(Wk));
    j = jn;
    tau = tau_new;
  }
  // c_q for the forecast at step i: sum_k (i - tau)^k / k! * W[k][q], k <= min(K, j)
  void coeffs(double i, float* c) const {
    const int ke = j < K ? j : K;
    double fact = 1.0, pw = 1.0;
    double acc[FF_MAX_K + 2] = {};
    for (int k = 0; k <= ke; ++k) {
      if (k > 0) { fact *= k; pw *= (i - tau); }
      for (int q = 0; q <= K; ++q) acc[q] += pw / fact * Wk[k][q];
    }
    for (int q = 0; q <= K; ++q) c[q] = (float)acc[q];
  }
};

// The layer actions of step i as a cached step: SITE where the mask is set in the paid
// modes, DRAFT elsewhere; in the recompute arm every layer after the first site is exact.
void cached_actions(const ff_plan& p, int i, int32_t* row) {
  const ff_sched_desc& s = p.s;
  const int L = p.L;
  const bool paid_mode = s.mode >= FF_VERIFY && s.mode != FF_DRAFT;
  bool paid_seen = false;
  for (int l = 0; l < L; ++l) {
    int a = paid_mode && p.mask[(size_t)i * L + l] ? FF_ACT_SITE : FF_ACT_DRAFT;
    if (s.mode == FF_RECOMPUTE && paid_seen) a = FF_ACT_RECOMPUTE;   // the rest of the step, exact
    paid_seen = paid_seen || a == FF_ACT_SITE;
    row[l] = a;
  }
}

// Row i of a plan: a refresh (ordinal j, written to slot j % S) or a cached step that
// reads the ring with the coefficients of cs at step i, with SITE where the mask is set
// in the paid modes.  cs must already hold the refreshes up to step i.
void plan_row(ff_plan* p, int i, bool refresh, int j, const CoefState& cs) {
  const ff_sched_desc& s = p->s;
  const int K = s.K, S = s.S, L = p->L;
  const int ke = j < K ? j : K;
  p->refresh_ord[i] = j;
  p->k_eff[i] = ke;
  for (int q = 0; q <= K; ++q) {
    p->read_slots[(size_t)i * (K + 1) + q] = -1;
    p->coeffs[(size_t)i * (K + 1) + q] = 0.f;
  }
  if (refresh) {
    p->step_kind[i] = FF_STEP_REFRESH;
    p->write_slot[i] = s.mode != FF_VANILLA ? j % S : -1;
    for (int l = 0; l < L; ++l) p->action[(size_t)i * L + l] = FF_ACT_EXACT;
    return;
  }
  p->step_kind[i] = FF_STEP_CACHED;
  p->write_slot[i] = -1;
  for (int q = 0; q <= ke; ++q) p->read_slots[(size_t)i * (K + 1) + q] = ((j - q) % S + S) % S;
  float c[FF_MAX_K + 2] = {};
  cs.coeffs((double)i, c);
  for (int q = 0; q <= ke; ++q) p->coeffs[(size_t)i * (K + 1) + q] = c[q];
  cached_actions(*p, i, &p->action[(size_t)i * L]);
}

// With history sums, the layers a run may cover: drafted layers off the site set.  A
// masked layer is a run of its own even in Draft, where it is drafted, so that Draft and
// Verify round their streams at the same layers and stay bitwise equal.
inline bool summable(const ff_plan& p, int i, int l, int32_t act) {
  return act == FF_ACT_DRAFT && !p.mask[(size_t)i * p.L + l];
}

// Maximal runs [l0, l1) of two or more summable layers on the steps that are, or (with an
// adaptive schedule) may become, cached steps: the runs a history sum can stand in for.
std::vector<std::pair<int, int>> plan_runs(const ff_plan& p) {
  std::vector<std::pair<int, int>> runs;
  const int L = p.L;
  std::vector<int32_t> row(L);
  for (int i = 1; i < p.s.T; ++i) {
    if (p.s.tau <= 0.f && p.step_kind[i] != FF_STEP_CACHED) continue;
    cached_actions(p, i, row.data());
    for (int l = 0; l < L;) {
      if (!summable(p, i, l, row[l])) { ++l; continue; }
      int l1 = l + 1;
      while (l1 < L && summable(p, i, l1, row[l1])) ++l1;
      if (l1 - l >= 2 && std::find(runs.begin(), runs.end(), std::make_pair(l, l1)) == runs.end())
        runs.emplace_back(l, l1);
      l = l1;
    }
  }
  return runs;
}

// the modes that forward (all or part of) the exact output of a paid site
bool forwards(int mode) { return mode == FF_FEATFIX || mode == FF_EXACT_ONLY || mode >= FF_TOKENS_PARTIAL; }

}  // namespace

namespace {

// Conditioning cache (ff_ctx_cond_cache).  The conditioning c_t = cond + TimeMLP(phi(1000 t_i))
// and every adaLN modulation vector depend on the class / text vector and the step only,
// never on the latent, so with the cache the context forms them for the whole schedule at
// step 0: the time embeddings and MLP of all T steps, SiLU(c_t) (bf16: as hi / lo rows),
// then one GEMM per weight set over the steps at which that layer runs exact, and the
// final layer's modulation for every step.  Layout of the caller's buffer (each part
// 256-byte aligned): PHI [T, 256], TMP and U [T, C] fp32; bf16: XS [T, 16 * groups, C]
// bf16, ZB (zeros, 6C bf16), OUT [T * 16 * groups, 6C] fp32 (the GEMM's hi / lo rows);
// fp32: CSA [T, B, C]; then per layer its modulation vectors [nb, B, ldy] fp32 and FMOD
// [T, B, 2C] fp32.
struct CondLayer { bool all; int nb; size_t off; int ldy; };
struct CondLayout {
  size_t PHI = 0, TMP = 0, U = 0, XS = 0, CSA = 0, ZB = 0, OUT = 0, FMOD = 0, total = 0;
  int R16 = 0;   // bf16: GEMM rows per step (16 per group of 8 model rows)
  std::vector<CondLayer> layer;
};

// Which steps' modulation a layer's GEMM covers: every step, or only the refresh steps
// (i % R == 0), the latter when the plan runs the layer exact at refresh steps only and
// the mask puts no site on it at a cached step.  The choice follows the mask, not the
// mode, so modes whose exact blocks coincide (FeatFix and Exact-only, Verify and Draft)
// read identical vectors; with tau > 0 every step may refresh.
bool cond_all_steps(const ff_plan& p, int l) {
  const int T = p.s.T, L = p.L, R = p.s.R;
  if (p.s.tau > 0.f) return true;
  for (int i = 0; i < T; ++i) {
    const int a = p.action[(size_t)i * L + l];
    const bool exact = a == FF_ACT_EXACT || a == FF_ACT_SITE || a == FF_ACT_RECOMPUTE;
    if (exact && i % R != 0) return true;
    if (p.step_kind[i] == FF_STEP_CACHED && p.mask[(size_t)i * L + l]) return true;
  }
  return false;
}

CondLayout cond_layout(const Model& m, const ff_plan& p) {
  CondLayout cl;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  const size_t T = p.s.T, C = m.C, B = m.B;
  const bool bf = m.dtype == FF_BF16;
  cl.R16 = 16 * ((m.B + 7) / 8);
  cl.PHI = take(T * FF_TEMB_DIM * 4);
  cl.TMP = take(T * C * 4);
  cl.U = take(T * C * 4);
  if (bf) {
    cl.XS = take(T * cl.R16 * C * 2);
    cl.ZB = take(6 * C * 2);
    cl.OUT = take(T * cl.R16 * 6 * C * 4);
  } else {
    cl.CSA = take(T * B * C * 4);
  }
  for (int l = 0; l < m.L; ++l) {
    CondLayer cy;
    cy.all = cond_all_steps(p, l);
    cy.nb = cy.all ? p.s.T : (p.s.T + p.s.R - 1) / p.s.R;
    cy.ldy = mod_floats(m.kinds[l], m.C);
    cy.off = take((size_t)cy.nb * B * cy.ldy * 4);
    cl.layer.push_back(cy);
  }
  cl.FMOD = take(T * B * 2 * C * 4);
  cl.total = off;
  return cl;
}

}  // namespace

struct ff_ctx {
  Model m;
  std::vector<ff_layer_weights> lw;
  ff_global_weights g;
  ff_plan plan;   // with tau > 0, row i is rewritten when step i is decided
  void* cache;
  void* ws;
  int next_step;
  std::vector<uint8_t> written;  // [L * S]: slot holds a refresh of this run
  std::vector<int32_t> realised; // [T]: kind of each step run, -1 before
  ff_counts counts;
  Prof prof;
  // adaptive refresh (tau > 0): refresh ordinal and recursion over the actual refresh
  // steps, the last refresh step, and the previous step's discrepancies on their way to
  // the host (pinned rel[L * B], event after the copy; checked: that step had sites)
  int a_j = -1, a_last = -1;
  CoefState a_cs{0};
  float* a_rel = nullptr;
  hipEvent_t a_ev = nullptr;
  bool a_checked = false;
  void* trace = nullptr;   // per-layer stream copies (ff_ctx_trace), [L][B*N*C]
  // history sums (ff_ctx_hist_sums): fp32 [runs][S][B*N*C], formed at every refresh
  float* hsum = nullptr;
  std::vector<std::pair<int, int>> runs;
  // conditioning cache (ff_ctx_cond_cache): formed at step 0 from cond, which every later
  // step must pass again
  char* cc = nullptr;
  CondLayout cc_lay;
  const float* cc_cond = nullptr;
  ~ff_ctx() {
    if (a_ev) (void)hipEventDestroy(a_ev);
    if (a_rel) (void)hipHostFree(a_rel);
  }
  void reset_adaptive() {
    a_j = -1;
    a_last = -1;
    a_cs = CoefState(plan.s.K);
    a_checked = false;
  }
};

namespace {

ff_status check_sched(const ff_sched_desc* s, int L) {
  if (!s) return fail(FF_E_NULL, "schedule descriptor is NULL");
  if (s->T < 1 || s->T > 100000) return fail(FF_E_RANGE, "T=%d out of range", s->T);
  if (s->R < 1) return fail(FF_E_RANGE, "R=%d must be >= 1", s->R);
  if (s->K < 0 || s->K > FF_MAX_K) return fail(FF_E_RANGE, "K=%d outside [0, %d]", s->K, FF_MAX_K);
  if (s->S < s->K + 1 || s->S > FF_MAX_SLOTS) return fail(FF_E_RANGE, "S=%d must be in [K+1, %d]", s->S, FF_MAX_SLOTS);
  if (s->mode < FF_VANILLA || s->mode > FF_RECOMPUTE) return fail(FF_E_RANGE, "mode=%d unknown", s->mode);
  if ((s->mode == FF_TOKENS_PARTIAL || s->mode == FF_CHANNELS_PARTIAL) && s->part_stride < 1)
    return fail(FF_E_RANGE, "part_stride=%d must be >= 1", s->part_stride);
  if (s->feature_mode != FF_RESIDUAL && s->feature_mode != FF_OUTPUT)
    return fail(FF_E_RANGE, "feature_mode=%d unknown", s->feature_mode);
  if (!(s->eps > 0.f)) return fail(FF_E_RANGE, "eps must be > 0");
  if (!(s->tau >= 0.f) || !std::isfinite(s->tau)) return fail(FF_E_RANGE, "tau must be finite and >= 0");
  if (s->tau > 0.f && s->mode != FF_VERIFY && s->mode != FF_FEATFIX)
    return fail(FF_E_RANGE, "tau > 0 needs the discrepancy of FF_VERIFY or FF_FEATFIX (mode %d)", s->mode);
  if (L < 1 || L > 4096) return fail(FF_E_RANGE, "n_layers=%d out of range", L);
  return FF_OK;
}

void build_plan(const ff_sched_desc& s, int L, const uint8_t* mask, ff_plan* p) {
  const int T = s.T, K = s.K;
  p->s = s;
  p->L = L;
  p->step_kind.assign(T, 0);
  p->refresh_ord.assign(T, 0);
  p->k_eff.assign(T, 0);
  p->read_slots.assign((size_t)T * (K + 1), -1);
  p->write_slot.assign(T, -1);
  p->action.assign((size_t)T * L, FF_ACT_EXACT);
  p->coeffs.assign((size_t)T * (K + 1), 0.f);
  p->mask.assign(mask, mask + (size_t)T * L);
  p->counts = ff_counts{0, 0, 0, 0};
  CoefState cs(K);
  int j = -1;
  for (int i = 0; i < T; ++i) {
    const bool refresh = s.mode == FF_VANILLA || i % s.R == 0;
    if (refresh) {
      ++j;
      cs.refresh((double)i);
    }
    plan_row(p, i, refresh, j, cs);
    if (refresh) {
      p->counts.n_full_refresh++;
      continue;
    }
    for (int l = 0; l < L; ++l) {
      const int a = p->action[(size_t)i * L + l];
      if (a == FF_ACT_RECOMPUTE) p->counts.n_recomputed++;
      if (a != FF_ACT_SITE) continue;
      p->counts.n_paid_checks++;
      if (forwards(s.mode)) p->counts.n_forwarded++;
    }
  }
}

ff_status check_terms(const Model& m, int n_slots, int layer, int k_eff, const int32_t* slots, const float* coeffs,
                      const void* cache, Terms* t) {
  if (!cache || !slots || !coeffs) return fail(FF_E_NULL, "cache, slots or coeffs is NULL");
  if (layer < 0 || layer >= m.L) return fail(FF_E_RANGE, "layer %d out of range", layer);
  if (n_slots < 1 || n_slots > FF_MAX_SLOTS) return fail(FF_E_RANGE, "n_slots %d out of range", n_slots);
  if (k_eff < 0 || k_eff > FF_MAX_K) return fail(FF_E_RANGE, "k_eff %d out of range", k_eff);
  t->n = k_eff + 1;
  const size_t slot_bytes = m.E() * m.es();
  for (int q = 0; q <= k_eff; ++q) {
    if (slots[q] < 0 || slots[q] >= n_slots) return fail(FF_E_RANGE, "slot %d out of range", slots[q]);
    t->slot[q] = reinterpret_cast<const char*>(cache) + ((size_t)layer * n_slots + slots[q]) * slot_bytes;
    t->c[q] = coeffs[q];
  }
  for (int q = k_eff + 1; q < kMaxTerms; ++q) { t->slot[q] = nullptr; t->c[q] = 0.f; }
  if (!aligned16(cache)) return fail(FF_E_SHAPE, "cache must be 16-byte aligned");
  return FF_OK;
}

// Argument checks shared by the two verify entry points (everything except the buffer
// that holds the partial sums).
ff_status check_verify(const ff_model_desc* m, const void* cache, int32_t n_slots, int32_t layer, int32_t k_eff,
                       const int32_t* slots, const float* coeffs, const void* u, const void* h_f, const void* h_out,
                       int32_t forward, int32_t stride, float eps, Model* md, Terms* t) {
  ff_status e = check_model(m, md);
  if (e) return e;
  if (!h_f || !h_out) return fail(FF_E_NULL, "h_f or h_out is NULL");
  e = check_terms(*md, n_slots, layer, k_eff, slots, coeffs, cache, t);
  if (e) return e;
  if (!(eps > 0.f)) return fail(FF_E_RANGE, "eps must be > 0");
  const size_t tb = md->E() * md->es();
  if ((const char*)h_out < (const char*)h_f + tb && (const char*)h_f < (const char*)h_out + tb)
    return fail(FF_E_SHAPE, "h_out overlaps h_f");
  if (!aligned16(h_f) || !aligned16(h_out) || (u && !aligned16(u))) return fail(FF_E_SHAPE, "pointers must be 16-byte aligned");
  if (forward < FF_FWD_DRAFT || forward > FF_FWD_CHANNELS) return fail(FF_E_RANGE, "forward=%d unknown", forward);
  if (forward >= FF_FWD_TOKENS && stride < 1) return fail(FF_E_RANGE, "stride=%d must be >= 1", stride);
  return FF_OK;
}

// Partial sums of ff_verify_replace_noalloc: a fixed device array per GPU (each device
// that loads the library holds its own copy until the process ends).  Host code never
// uses the array's name as an address: the address of the current device's copy comes
// from hipGetSymbolAddress, once per device, and is kept here.
constexpr size_t kScratchFloats = (size_t)FF_NOALLOC_VERIFY_MAX_B * 2048 * 2;
static __device__ __align__(256) float scratch[kScratchFloats];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

ff_status scratch_of_current_device(float** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev), "no-allocation verify: current device");
  if (dev < 0 || dev >= kMaxDevices) return fail(FF_E_UNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "no-allocation verify: scratch address");
    if (!p) return fail(FF_E_HIP, "no-allocation verify: scratch address is NULL");
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_ptr[dev];
  return FF_OK;
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

int32_t ff_abi_version(void) { return FF_ABI_VERSION; }

const char* ff_last_error(void) { return g_err; }

ff_status ff_plan_build(const ff_sched_desc* s, int32_t n_layers, const uint8_t* site_mask, ff_plan** out) {
  try {
    if (!out || !site_mask) return fail(FF_E_NULL, "out or site_mask is NULL");
    ff_status e = check_sched(s, n_layers);
    if (e) return e;
    ff_plan* p = new ff_plan();
    build_plan(*s, n_layers, site_mask, p);
    *out = p;
    return ok();
  } catch (const std::bad_alloc&) {
    return fail(FF_E_UNSUPPORTED, "out of host memory");
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

void ff_plan_destroy(ff_plan* p) { delete p; }

ff_status ff_plan_export(const ff_plan* p, int32_t* step_kind, int32_t* refresh_ord, int32_t* k_eff,
                         int32_t* read_slots, int32_t* write_slot, int32_t* action, float* coeffs,
                         ff_counts* counts) {
  if (!p) return fail(FF_E_NULL, "plan is NULL");
  const size_t T = p->s.T;
  if (step_kind) memcpy(step_kind, p->step_kind.data(), T * 4);
  if (refresh_ord) memcpy(refresh_ord, p->refresh_ord.data(), T * 4);
  if (k_eff) memcpy(k_eff, p->k_eff.data(), T * 4);
  if (read_slots) memcpy(read_slots, p->read_slots.data(), p->read_slots.size() * 4);
  if (write_slot) memcpy(write_slot, p->write_slot.data(), T * 4);
  if (action) memcpy(action, p->action.data(), p->action.size() * 4);
  if (coeffs) memcpy(coeffs, p->coeffs.data(), p->coeffs.size() * 4);
  if (counts) *counts = p->counts;
  return ok();
}

size_t ff_cache_bytes(const ff_model_desc* m, int32_t n_slots) {
  Model md;
  if (check_model(m, &md) != FF_OK || n_slots < 1) return 0;
  return (size_t)md.L * n_slots * md.E() * md.es();
}

size_t ff_workspace_bytes(const ff_model_desc* m) {
  Model md;
  if (check_model(m, &md) != FF_OK) return 0;
  return ws_layout(md).total;
}

ff_status ff_block_exact(const ff_model_desc* m, int32_t layer, const ff_layer_weights* w, const float* c_t,
                         const void* u, void* h, void* ws, size_t ws_bytes, ff_stream_t stream) {
  try {
    Model md;
    ff_status e = check_model(m, &md);
    if (e) return e;
    if (layer < 0 || layer >= md.L) return fail(FF_E_RANGE, "layer %d out of range [0, %d)", layer, md.L);
    if (!c_t || !u || !h || !ws) return fail(FF_E_NULL, "c_t, u, h or ws is NULL");
    e = check_layer_weights(w, md.kinds[layer], layer);
    if (e) return e;
    const Ws L = ws_layout(md);
    if (ws_bytes < L.total) return fail(FF_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);
    if (!aligned16(u) || !aligned16(h) || !aligned16(ws) || !aligned16(c_t))
      return fail(FF_E_SHAPE, "device pointers must be 16-byte aligned");
    const size_t tb = md.E() * md.es();
    const char *pu = (const char*)u, *ph = (const char*)h, *pw = (const char*)ws;
    if ((ph < pu + tb && pu < ph + tb) || (ph < pw + L.total && pw < ph + tb))
      return fail(FF_E_SHAPE, "h overlaps u or the workspace");
    Exec ex{reinterpret_cast<hipStream_t>(stream), nullptr, md.dtype, md.es()};
    float* cs = at<float>(ws, L.CS);
    HIP_TRY(silu_rows(c_t, cs, md.B, md.C, nullptr, ex.st), "block: silu(c_t)");
    e = exec_block(md, md.kinds[layer], *w, cs, u, h, ws, ex);
    if (e) return e;
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

ff_status ff_cache_update(const ff_model_desc* m, void* cache, int32_t n_slots, int32_t layer, int32_t slot,
                          const void* u, const void* h, int32_t feature_mode, ff_stream_t stream) {
  Model md;
  ff_status e = check_model(m, &md);
  if (e) return e;
  if (!cache || !h) return fail(FF_E_NULL, "cache or h is NULL");
  if (feature_mode != FF_RESIDUAL && feature_mode != FF_OUTPUT) return fail(FF_E_RANGE, "feature_mode unknown");
  if (feature_mode == FF_RESIDUAL && !u) return fail(FF_E_NULL, "u is NULL in residual mode");
  if (layer < 0 || layer >= md.L) return fail(FF_E_RANGE, "layer %d out of range", layer);
  if (n_slots < 1 || n_slots > FF_MAX_SLOTS || slot < 0 || slot >= n_slots)
    return fail(FF_E_RANGE, "slot %d / n_slots %d out of range", slot, n_slots);
  if (!aligned16(cache) || !aligned16(h) || (u && !aligned16(u))) return fail(FF_E_SHAPE, "pointers must be 16-byte aligned");
  void* dst = (char*)cache + ((size_t)layer * n_slots + slot) * md.E() * md.es();
  HIP_TRY(ff::cache_update(md.dtype, dst, feature_mode == FF_RESIDUAL ? u : nullptr, h, md.E(),
                           reinterpret_cast<hipStream_t>(stream)), "cache update");
  return ok();
}

ff_status ff_draft_forecast(const ff_model_desc* m, const void* cache, int32_t n_slots, int32_t layer, int32_t k_eff,
                            const int32_t* slots, const float* coeffs, const void* u, void* h_d, ff_stream_t stream) {
  Model md;
  ff_status e = check_model(m, &md);
  if (e) return e;
  if (!h_d) return fail(FF_E_NULL, "h_d is NULL");
  Terms t{};
  e = check_terms(md, n_slots, layer, k_eff, slots, coeffs, cache, &t);
  if (e) return e;
  if (!aligned16(h_d) || (u && !aligned16(u))) return fail(FF_E_SHAPE, "pointers must be 16-byte aligned");
  HIP_TRY(ff::draft(md.dtype, t, u, h_d, md.E(), reinterpret_cast<hipStream_t>(stream)), "draft");
  return ok();
}

ff_status ff_verify_replace(const ff_model_desc* m, const void* cache, int32_t n_slots, int32_t layer, int32_t k_eff,
                            const int32_t* slots, const float* coeffs, const void* u, const void* h_f, void* h_out,
                            int32_t forward, int32_t stride, float eps, float* rel_l1, void* ws, size_t ws_bytes,
                            ff_stream_t stream) {
  Model md;
  Terms t{};
  ff_status e = check_verify(m, cache, n_slots, layer, k_eff, slots, coeffs, u, h_f, h_out, forward, stride, eps,
                             &md, &t);
  if (e) return e;
  if (!ws) return fail(FF_E_NULL, "ws is NULL");
  const Ws L = ws_layout(md);
  if (ws_bytes < L.total) return fail(FF_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);
  const Forward fw{forward, stride, md.C};
  HIP_TRY(ff::verify(md.dtype, t, u, h_f, h_out, fw, md.B, (size_t)md.N * md.C, eps, rel_l1,
                     at<float>(ws, L.PART), reinterpret_cast<hipStream_t>(stream)), "verify");
  return ok();
}

ff_status ff_verify_replace_noalloc(const ff_model_desc* m, const void* cache, int32_t n_slots, int32_t layer,
                                    int32_t k_eff, const int32_t* slots, const float* coeffs, const void* u,
                                    const void* h_f, void* h_out, int32_t forward, int32_t stride, float eps,
                                    float* rel_l1, ff_stream_t stream) {
  try {
    Model md;
    Terms t{};
    ff_status e = check_verify(m, cache, n_slots, layer, k_eff, slots, coeffs, u, h_f, h_out, forward, stride, eps,
                               &md, &t);
    if (e) return e;
    if (md.B > FF_NOALLOC_VERIFY_MAX_B || verify_partials_floats(md.B) > kScratchFloats)
      return fail(FF_E_WORKSPACE, "no-allocation verify takes B <= %d (B = %d)", FF_NOALLOC_VERIFY_MAX_B, md.B);
    float* part = nullptr;
    e = scratch_of_current_device(&part);
    if (e) return e;
    const Forward fw{forward, stride, md.C};
    HIP_TRY(ff::verify(md.dtype, t, u, h_f, h_out, fw, md.B, (size_t)md.N * md.C, eps, rel_l1, part,
                       reinterpret_cast<hipStream_t>(stream)), "verify (no allocation)");
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

ff_status ff_ctx_create(const ff_model_desc* m, const ff_layer_weights* layer_w, const ff_global_weights* g,
                        const ff_plan* p, void* cache, size_t cache_bytes, void* ws, size_t ws_bytes, ff_ctx** out) {
  try {
    if (!out) return fail(FF_E_NULL, "out is NULL");
    Model md;
    ff_status e = check_model(m, &md);
    if (e) return e;
    const bool vanilla = p && p->s.mode == FF_VANILLA;   // Vanilla never touches the history
    if (!layer_w || !g || !p || (!cache && !vanilla) || !ws) return fail(FF_E_NULL, "weights, plan, cache or ws is NULL");
    if (p->L != md.L) return fail(FF_E_SHAPE, "plan has %d layers, model %d", p->L, md.L);
    for (int l = 0; l < md.L; ++l) {
      e = check_layer_weights(&layer_w[l], md.kinds[l], l);
      if (e) return e;
    }
    if (!g->t1_w || !g->t1_b || !g->t2_w || !g->t2_b || !g->pe_w || !g->pe_b || !g->fmod_w || !g->fmod_b ||
        !g->f_w || !g->f_b)
      return fail(FF_E_NULL, "a global weight pointer is NULL");
    const size_t need_cache = vanilla ? 0 : (size_t)md.L * p->s.S * md.E() * md.es();
    if (cache_bytes < need_cache) return fail(FF_E_WORKSPACE, "cache %zu < %zu bytes", cache_bytes, need_cache);
    const Ws L = ws_layout(md);
    if (ws_bytes < L.total) return fail(FF_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);
    if ((cache && !aligned16(cache)) || !aligned16(ws)) return fail(FF_E_SHAPE, "cache and ws must be 16-byte aligned");
    ff_ctx* c = new ff_ctx();
    c->m = md;
    c->lw.assign(layer_w, layer_w + md.L);
    c->g = *g;
    c->plan = *p;
    c->cache = cache;
    c->ws = ws;
    c->next_step = 0;
    c->written.assign((size_t)md.L * p->s.S, 0);
    c->realised.assign(p->s.T, -1);
    c->counts = ff_counts{0, 0, 0, 0};
    c->reset_adaptive();
    if (p->s.tau > 0.f) {
      hipError_t he = hipHostMalloc((void**)&c->a_rel, (size_t)md.L * md.B * sizeof(float), hipHostMallocDefault);
      if (he == hipSuccess) he = hipEventCreateWithFlags(&c->a_ev, hipEventDisableTiming);
      if (he != hipSuccess) {
        delete c;
        return fail(FF_E_HIP, "adaptive refresh buffers: %s", hipGetErrorString(he));
      }
    }
    *out = c;
    return ok();
  } catch (const std::bad_alloc&) {
    return fail(FF_E_UNSUPPORTED, "out of host memory");
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

void ff_ctx_destroy(ff_ctx* c) { delete c; }

ff_status ff_ctx_reset(ff_ctx* c) {
  if (!c) return fail(FF_E_NULL, "ctx is NULL");
  c->next_step = 0;
  std::fill(c->written.begin(), c->written.end(), 0);
  std::fill(c->realised.begin(), c->realised.end(), -1);
  c->counts = ff_counts{0, 0, 0, 0};
  c->reset_adaptive();
  return ok();
}

ff_status ff_ctx_step_kinds(const ff_ctx* c, int32_t* kinds) {
  if (!c || !kinds) return fail(FF_E_NULL, "ctx or kinds is NULL");
  memcpy(kinds, c->realised.data(), c->realised.size() * sizeof(int32_t));
  return ok();
}

ff_status ff_get_counts(const ff_ctx* c, ff_counts* out) {
  if (!c || !out) return fail(FF_E_NULL, "ctx or out is NULL");
  *out = c->counts;
  return ok();
}

namespace {

// The conditioning of every step of c's schedule into its cache (CondLayout): the same
// time embedding, time MLP and SiLU as each step forms, for all T steps at once, then each
// layer's modulation as one GEMM over the steps it needs and the final layer's for all.
// bf16: SiLU(c_t) enters the GEMM as bf16 hi / lo rows (the split the GEMVs use), whose two
// products are summed with the bias afterwards; fp32: the fp32 rows directly.
ff_status cond_precompute(ff_ctx* c, const float* cond, Exec& ex) {
  const Model& m = c->m;
  const CondLayout& cl = c->cc_lay;
  const int T = c->plan.s.T, R = c->plan.s.R, C = m.C, B = m.B;
  const bool bf = m.dtype == FF_BF16;
  char* base = c->cc;
  hipStream_t st = ex.st;
  float* phi = reinterpret_cast<float*>(base + cl.PHI);
  float* tmp = reinterpret_cast<float*>(base + cl.TMP);
  float* u = reinterpret_cast<float*>(base + cl.U);
  HIP_TRY(ex.other((double)T * FF_TEMB_DIM * 4, [&] { return time_embed_steps((double)T, T, phi, st); }),
          "conditioning cache: time embedding");
  for (int r0 = 0; r0 < T; r0 += kGemvMaxB) {
    const int nr = std::min(kGemvMaxB, T - r0);
    GemvArgs g1{phi + (size_t)r0 * FF_TEMB_DIM, FF_TEMB_DIM, 0, c->g.t1_w, c->g.t1_b, C, FF_TEMB_DIM, nr,
                tmp + (size_t)r0 * C, C, 1, nullptr, 0};
    HIP_TRY(ex.gemv(g1), "conditioning cache: time mlp 1");
    GemvArgs g2{tmp + (size_t)r0 * C, C, 0, c->g.t2_w, c->g.t2_b, C, C, nr, u + (size_t)r0 * C, C, 0, nullptr, 0};
    HIP_TRY(ex.gemv(g2), "conditioning cache: time mlp 2");
  }
  uint16_t* xs = bf ? reinterpret_cast<uint16_t*>(base + cl.XS) : nullptr;
  float* csa = bf ? nullptr : reinterpret_cast<float*>(base + cl.CSA);
  uint16_t* zb = bf ? reinterpret_cast<uint16_t*>(base + cl.ZB) : nullptr;
  HIP_TRY(ex.other((double)T * B * C * 8, [&] { return cond_split(u, cond, T, B, C, xs, csa, zb, bf ? 6 * C : 0, st); }),
          "conditioning cache: silu(c_t)");
  float* out = bf ? reinterpret_cast<float*>(base + cl.OUT) : nullptr;
  // one weight set over nb step blocks (every step, or every R-th) -> dst [nb, B, ldy]
  auto modulate = [&](const void* W, const void* bias, int N, bool all, int nb, float* dst, int ldy) -> ff_status {
    if (bf) {
      const int M = nb * cl.R16;
      const RowMap am = all ? RowMap{M, M, 0} : RowMap{cl.R16, cl.R16 * R, 0};
      GemmArgs g = gemm_args(xs, C, am, W, zb, M, N, C, EPI_BIAS, out, N, RowMap{M, M, 0});
      g.out_f32 = 1;
      HIP_TRY(ex.mod_gemm(g), "conditioning cache: modulation");
      HIP_TRY(ex.other(((double)M + nb * B) * N * 4.0,
                       [&] { return mod_combine(m.dtype, out, N, bias, dst, ldy, nb, B, st); }),
              "conditioning cache: modulation sum");
    } else {
      const int M = nb * B;
      const RowMap am = all ? RowMap{M, M, 0} : RowMap{B, B * R, 0};
      GemmArgs g = gemm_args(csa, C, am, W, bias, M, N, C, EPI_BIAS, dst, ldy, RowMap{M, M, 0});
      HIP_TRY(ex.mod_gemm(g), "conditioning cache: modulation");
    }
    return FF_OK;
  };
  for (int l = 0; l < m.L; ++l) {
    const CondLayer& cy = cl.layer[l];
    float* dst = reinterpret_cast<float*>(base + cy.off);
    const ff_stream_weights* sw = c->lw[l].s;
    const int kind = m.kinds[l];
    const int N = kind == FF_MMDIT_SINGLE ? 3 * C : 6 * C;
    ff_status e = modulate(sw[0].mod_w, sw[0].mod_b, N, cy.all, cy.nb, dst, cy.ldy);
    if (!e && kind == FF_MMDIT_DOUBLE) e = modulate(sw[1].mod_w, sw[1].mod_b, N, cy.all, cy.nb, dst + 6 * C, cy.ldy);
    if (e) return e;
  }
  return modulate(c->g.fmod_w, c->g.fmod_b, 2 * C, true, T, reinterpret_cast<float*>(base + cl.FMOD), 2 * C);
}

}  // namespace

ff_status ff_denoise_step(ff_ctx* c, int32_t step, float* x, const float* cond, const void* txt, float* audit,
                          ff_stream_t stream) {
  try {
    if (!c || !x || !cond) return fail(FF_E_NULL, "ctx, x or cond is NULL");
    const Model& m = c->m;
    const ff_plan& p = c->plan;
    const ff_sched_desc& s = p.s;
    if (m.n_txt > 0 && !txt) return fail(FF_E_NULL, "txt is NULL but n_txt = %d", m.n_txt);
    if (step != c->next_step || step >= s.T)
      return fail(FF_E_STATE, "step %d out of order (expected %d of %d)", step, c->next_step, s.T);
    if (!aligned16(x) || !aligned16(cond) || (txt && !aligned16(txt))) return fail(FF_E_SHAPE, "pointers must be 16-byte aligned");
    if (c->cc && step > 0 && cond != c->cc_cond)
      return fail(FF_E_STATE, "step %d: cond is not the buffer the conditioning cache was formed from at step 0", step);
    const int L = m.L, K = s.K, S = s.S, i = step;
    if (s.tau > 0.f) {
      // adaptive refresh: decide this step from the interval and the previous step's
      // largest site discrepancy, then write row i of the context's plan
      bool refresh = i == 0 || i - c->a_last >= s.R;
      if (!refresh && c->a_checked) {
        HIP_TRY(hipEventSynchronize(c->a_ev), "adaptive refresh: discrepancy copy");
        float dmax = 0.f;
        bool nan = false;
        for (int l = 0; l < L; ++l) {
          if (c->plan.action[(size_t)(i - 1) * L + l] != FF_ACT_SITE) continue;
          for (int b = 0; b < m.B; ++b) {
            const float d = c->a_rel[(size_t)l * m.B + b];
            if (d != d) nan = true;
            else dmax = std::max(dmax, d);
          }
        }
        refresh = nan || !(dmax <= s.tau);
      }
      if (refresh) {
        c->a_j++;
        c->a_cs.refresh((double)i);
        c->a_last = i;
      }
      plan_row(&c->plan, i, refresh, c->a_j, c->a_cs);
    }
    // host-side state checks first: nothing is launched if the plan would read an unwritten slot
    if (p.step_kind[i] == FF_STEP_CACHED) {
      for (int l = 0; l < L; ++l) {
        if (p.action[(size_t)i * L + l] == FF_ACT_EXACT || p.action[(size_t)i * L + l] == FF_ACT_RECOMPUTE) continue;
        if (s.mode == FF_EXACT_ONLY && p.action[(size_t)i * L + l] == FF_ACT_SITE) continue;
        for (int q = 0; q <= p.k_eff[i]; ++q) {
          const int sl = p.read_slots[(size_t)i * (K + 1) + q];
          if (sl < 0 || !c->written[(size_t)l * S + sl])
            return fail(FF_E_STATE, "step %d layer %d reads slot %d that holds no refresh", i, l, sl);
        }
      }
    }
    Exec ex{reinterpret_cast<hipStream_t>(stream), &c->prof, m.dtype, m.es()};
    hipStream_t st = ex.st;
    const Ws W = ws_layout(m);
    void* ws = c->ws;
    const int C = m.C, dt = m.dtype;
    const size_t es = m.es(), E = m.E(), tb = E * es;
    const double T = s.T;
    const double t_i = 1.0 - i / T, t_n = 1.0 - (i + 1) / T;
    float* phi = at<float>(ws, W.PHI);
    float* tmp = at<float>(ws, W.TMP);
    float* ct = at<float>(ws, W.CT);
    float* cs = at<float>(ws, W.CS);
    uint16_t* xs = dt == FF_BF16 ? at<uint16_t>(ws, W.XS) : nullptr;
    const CondLayout& cl = c->cc_lay;
    if (c->cc && i == 0) {   // the conditioning of the whole schedule (cond is checked at later steps)
      if (ff_status e = cond_precompute(c, cond, ex)) return e;
      c->cc_cond = cond;
    }
    if (!c->cc) {
      // conditioning: c_t = cond + W_t2 SiLU(W_t1 phi(1000 t) + b_t1) + b_t2
      HIP_TRY(ex.other(FF_TEMB_DIM * 4.0, [&] { return time_embed(1000.0 * t_i, phi, st); }), "time embedding");
      GemvArgs g1{phi, 0, 0, c->g.t1_w, c->g.t1_b, C, FF_TEMB_DIM, m.B, tmp, C, 1, nullptr, 0};
      HIP_TRY(ex.gemv(g1), "time mlp 1");
      GemvArgs g2{tmp, C, 0, c->g.t2_w, c->g.t2_b, C, C, m.B, ct, C, 0, cond, C};
      HIP_TRY(ex.gemv(g2), "time mlp 2");
      // bf16: SiLU(c_t) also as the hi / lo split that the modulation batches and the final
      // modulation read (made once here rather than by each of their workgroups)
      HIP_TRY(ex.other(8.0 * m.B * C, [&] { return silu_rows(ct, cs, m.B, C, xs, st); }), "silu(c_t)");
    }
    // Modulation of the layers that run exact this step, computed kModLayers layers at a
    // time in one batched GEMV launch each; mod_of[l] = that layer's vectors.
    auto runs_exact = [&](int l) {
      const int a = p.action[(size_t)i * L + l];
      return a == FF_ACT_EXACT || a == FF_ACT_SITE || a == FF_ACT_RECOMPUTE;
    };
    float* mods = at<float>(ws, W.MODS);
    std::vector<const float*> mod_of(L, nullptr);
    auto ensure_mod = [&](int l) -> ff_status {
      if (mod_of[l]) return FF_OK;
      if (c->cc) {   // formed at step 0
        const CondLayer& cy = cl.layer[l];
        if (!cy.all && i % s.R) return fail(FF_E_STATE, "step %d layer %d: no cached modulation", i, l);
        mod_of[l] = reinterpret_cast<const float*>(c->cc + cy.off) + (size_t)(cy.all ? i : i / s.R) * m.B * cy.ldy;
        return FF_OK;
      }
      GemvBatch bt{};
      bt.x = cs; bt.ldx = C; bt.silu_in = 0; bt.K = C; bt.B = m.B; bt.xs = xs;
      int slot = 0;
      for (int l2 = l; l2 < L && slot < kModLayers; ++l2) {
        if (!runs_exact(l2)) continue;
        float* dst = mods + (size_t)slot * W.mod_slot;
        const int kind = m.kinds[l2];
        const ff_stream_weights* sw = c->lw[l2].s;
        if (kind == FF_MMDIT_SINGLE) {
          bt.job[bt.njobs++] = GemvJob{sw[0].mod_w, sw[0].mod_b, dst, 3 * C, 3 * C};
        } else if (kind == FF_MMDIT_DOUBLE) {
          bt.job[bt.njobs++] = GemvJob{sw[0].mod_w, sw[0].mod_b, dst, 6 * C, 12 * C};
          bt.job[bt.njobs++] = GemvJob{sw[1].mod_w, sw[1].mod_b, dst + 6 * C, 6 * C, 12 * C};
        } else {
          bt.job[bt.njobs++] = GemvJob{sw[0].mod_w, sw[0].mod_b, dst, 6 * C, 6 * C};
        }
        mod_of[l2] = dst;
        ++slot;
      }
      HIP_TRY(ex.gemv_batch(bt), "batched modulation");
      return FF_OK;
    };
    // tokens: X = [txt ; patch_embed(patchify(x))]
    PatchGeom pg{m.B, m.lat_c, m.lat_f, m.lat_h, m.lat_w, m.pt, m.ph, m.pw};
    if (m.cfg) {   // guided pairs: rows b and b + B/2 read latent b; the Euler step combines them
      pg.lat_B = m.B / 2;
      pg.cfg_half = m.B / 2;
      pg.cfg_scale = m.cfg_scale;
    }
    void* patches = at(ws, W.PATCH);
    const double lat_elems = (double)m.B * m.n_img * m.P;
    void* cur = at(ws, W.X0);
    void* alt = at(ws, W.X1);
    const RowMap img{m.n_img, m.N, m.n_txt};
    const RowMap ident{m.B * m.n_img, m.B * m.n_img, 0};
    HIP_TRY(ex.other(lat_elems * (4 + es), [&] { return patchify(dt, x, patches, pg, st); }), "patchify");
    GemmArgs pe = gemm_args(patches, m.P, ident, c->g.pe_w, c->g.pe_b, m.B * m.n_img, C, m.P, EPI_BIAS, cur, C, img);
    HIP_TRY(ex.gemm(pe), "patch embed");
    if (m.n_txt > 0)
      HIP_TRY(ex.other(2.0 * m.B * m.n_txt * C * es, [&] { return copy_rows(dt, txt, cur, m.B, m.n_txt, m.N, 0, C, st); }),
              "text rows");
    // layers by the plan
    const int mode = s.mode;
    const bool resid = s.feature_mode == FF_RESIDUAL;
    // with a trace buffer, the stream after layer l (in cur) is copied to its slot
    auto trace_to = [&](int l) -> ff_status {
      if (c->trace)
        HIP_TRY(hipMemcpyAsync((char*)c->trace + (size_t)l * tb, cur, tb, hipMemcpyDeviceToDevice, st), "trace copy");
      return FF_OK;
    };
    // a run of drafted layers applied from history sums and followed by a paid site is
    // left to that site block's first LayerNorm (one pass fewer over the stream)
    Terms pending{};
    const Terms* defer = nullptr;
    for (int l = 0; l < L; ++l) {
      const int act = p.action[(size_t)i * L + l];
      if (act == FF_ACT_EXACT) {
        ff_status e = ensure_mod(l);
        if (e) return e;
        // bf16: the refresh is fused into the block's last GEMM; fp32: a separate pass
        void* dst = mode != FF_VANILLA ? (char*)c->cache + ((size_t)l * S + p.write_slot[i]) * tb : nullptr;
        const bool fuse = dst && dt == FF_BF16;
        e = exec_block(m, m.kinds[l], c->lw[l], cs, cur, alt, ws, ex, mod_of[l], fuse ? dst : nullptr, resid);
        if (e) return e;
        if (dst && !fuse) HIP_TRY(ex.cache(dst, resid ? cur : nullptr, alt, E), "cache update");
        void* t = cur; cur = alt; alt = t;
        if (ff_status te = trace_to(l)) return te;
        continue;
      }
      if (act == FF_ACT_RECOMPUTE) {   // the recompute arm: the exact block, no history refresh
        ff_status e = ensure_mod(l);
        if (e) return e;
        e = exec_block(m, m.kinds[l], c->lw[l], cs, cur, alt, ws, ex, mod_of[l]);
        if (e) return e;
        void* t = cur; cur = alt; alt = t;
        if (ff_status te = trace_to(l)) return te;
        continue;
      }
      if (act == FF_ACT_SITE && mode == FF_EXACT_ONLY) {
        ff_status e = ensure_mod(l);
        if (e) return e;
        e = exec_block(m, m.kinds[l], c->lw[l], cs, cur, alt, ws, ex, mod_of[l], nullptr, true, defer);
        defer = nullptr;
        if (e) return e;
        void* t = cur; cur = alt; alt = t;
        if (ff_status te = trace_to(l)) return te;
        continue;
      }
      Terms tm{};
      tm.n = p.k_eff[i] + 1;
      for (int q = 0; q < tm.n; ++q) {
        const int sl = p.read_slots[(size_t)i * (K + 1) + q];
        tm.slot[q] = (const char*)c->cache + ((size_t)l * S + sl) * tb;
        tm.c[q] = p.coeffs[(size_t)i * (K + 1) + q];
      }
      if (act == FF_ACT_DRAFT) {
        // the maximal run of drafted layers starting here, applied in one pass (same bits);
        // layer by layer while tracing
        int l2 = l + 1;
        if (c->hsum && !summable(p, i, l, act)) {
          // a masked layer in Draft: drafted alone, as Verify's site drafts it
        } else if (c->hsum) {
          while (!c->trace && l2 < L && summable(p, i, l2, p.action[(size_t)i * L + l2])) ++l2;
        } else {
          while (!c->trace && l2 < L && p.action[(size_t)i * L + l2] == FF_ACT_DRAFT) ++l2;
        }
        int r = -1;
        if (c->hsum && resid && l2 - l >= 2)
          for (int q = 0; q < (int)c->runs.size(); ++q)
            if (c->runs[q] == std::make_pair(l, l2)) r = q;
        if (r >= 0) {   // the run from its history sums (formed at the refreshes)
          Terms ts = tm;
          for (int q = 0; q < ts.n; ++q)
            ts.slot[q] = c->hsum + ((size_t)r * S + p.read_slots[(size_t)i * (K + 1) + q]) * E;
          if (l2 < L && p.action[(size_t)i * L + l2] == FF_ACT_SITE) {
            pending = ts;
            defer = &pending;
          } else {
            HIP_TRY(ex.draft_sum(ts, cur, E), "draft from history sums");
          }
        } else if (l2 - l == 1) {
          HIP_TRY(ex.draft(tm, resid ? cur : nullptr, cur, E), "draft");
        } else {
          HIP_TRY(ex.draft_run(tm, l2 - l, (size_t)S * E, resid, cur, E), "draft run");
        }
        l = l2 - 1;
        if (ff_status te = trace_to(l)) return te;
        continue;
      }
      // paid site: exact output from the same incoming state, then verify + forward
      void* hf = at(ws, W.HF);
      ff_status e = ensure_mod(l);
      if (e) return e;
      e = exec_block(m, m.kinds[l], c->lw[l], cs, cur, hf, ws, ex, mod_of[l], nullptr, true, defer);
      defer = nullptr;
      if (e) return e;
      float* rel = audit ? audit + ((size_t)i * L + l) * m.B
                         : s.tau > 0.f ? at<float>(ws, W.REL) + (size_t)l * m.B : nullptr;
      const Forward fw{mode == FF_VERIFY ? FWD_DRAFT
                       : mode == FF_TOKENS_PARTIAL ? FWD_TOKENS
                       : mode == FF_CHANNELS_PARTIAL ? FWD_CHANNELS : FWD_EXACT,
                       s.part_stride, C};
      HIP_TRY(ex.verify(tm, resid ? cur : nullptr, hf, cur, fw, m.B, (size_t)m.N * C, s.eps,
                        rel, at<float>(ws, W.PART)), "verify");
      if (ff_status te = trace_to(l)) return te;
    }
    // a refresh rewrote slot write_slot of every layer: re-form each run's sum of it
    if (c->hsum && p.step_kind[i] == FF_STEP_REFRESH && mode != FF_VANILLA) {
      const int ws_i = p.write_slot[i];
      for (size_t r = 0; r < c->runs.size(); ++r) {
        const int l0 = c->runs[r].first, n = c->runs[r].second - l0;
        HIP_TRY(ex.hist_sum((const char*)c->cache + ((size_t)l0 * S + ws_i) * tb, n, (size_t)S * E,
                            c->hsum + (r * S + ws_i) * E, E), "history sums");
      }
    }
    // final layer on the image rows, unpatchify and Euler
    float* mod = at<float>(ws, W.MOD);
    if (c->cc) {
      mod = reinterpret_cast<float*>(c->cc + cl.FMOD) + (size_t)i * m.B * 2 * C;
    } else {
      GemvArgs gf{cs, C, 0, c->g.fmod_w, c->g.fmod_b, 2 * C, C, m.B, mod, 2 * C, 0, nullptr, 0, xs};
      HIP_TRY(ex.gemv(gf), "final modulation");
    }
    if (final_layer_ok(dt, m.P, C) && !m.cfg) {
      // LN + modulation + final linear + unpatchify + Euler in one launch, one wavefront
      // per image token (small final weights only)
      const FinalArgs fa{cur, C, img, m.B * m.n_img, C, m.ln_eps, mod, mod + C, 2 * C, c->g.f_w, c->g.f_b,
                         x, (float)(t_n - t_i), pg};
      HIP_TRY(ex.other((double)m.B * m.n_img * C * es + lat_elems * 8.0, [&] { return final_layer(dt, fa, st); }),
              "final layer");
    } else {
      void* lna = at(ws, W.LNA);
      LnModArgs ln{cur, 0, C, img, m.B * m.n_img, C, m.ln_eps, mod, mod + C, 2 * C, lna, C};
      HIP_TRY(ex.ln(ln), "final ln");
      float* yf = at<float>(ws, W.YF);
      GemmArgs gfl = gemm_args(lna, C, img, c->g.f_w, c->g.f_b, m.B * m.n_img, m.P, C, EPI_BIAS, yf, m.P, ident);
      gfl.out_f32 = 1;
      HIP_TRY(ex.gemm(gfl), "final linear");
      HIP_TRY(ex.other(lat_elems * 12.0, [&] { return unpatchify_euler(yf, x, (float)(t_n - t_i), pg, st); }),
              "unpatchify + euler");
    }
    // bookkeeping after a successful enqueue
    if (s.tau > 0.f) {
      // this step's site discrepancies go to the host for the next step's decision
      c->a_checked = false;
      for (int l = 0; l < L; ++l) c->a_checked |= p.action[(size_t)i * L + l] == FF_ACT_SITE;
      if (c->a_checked) {
        const float* src = audit ? audit + (size_t)i * L * m.B : at<float>(ws, W.REL);
        HIP_TRY(hipMemcpyAsync(c->a_rel, src, (size_t)L * m.B * sizeof(float), hipMemcpyDeviceToHost, st),
                "adaptive refresh: discrepancy copy");
        HIP_TRY(hipEventRecord(c->a_ev, st), "adaptive refresh: event");
      }
    }
    c->realised[i] = p.step_kind[i];
    if (p.step_kind[i] == FF_STEP_REFRESH) {
      c->counts.n_full_refresh++;
      if (mode != FF_VANILLA)
        for (int l = 0; l < L; ++l) c->written[(size_t)l * S + p.write_slot[i]] = 1;
    } else {
      for (int l = 0; l < L; ++l) {
        const int a = p.action[(size_t)i * L + l];
        if (a == FF_ACT_RECOMPUTE) c->counts.n_recomputed++;
        if (a != FF_ACT_SITE) continue;
        c->counts.n_paid_checks++;
        if (forwards(mode)) c->counts.n_forwarded++;
      }
    }
    c->next_step++;
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

size_t ff_hist_sum_bytes(const ff_model_desc* m, const ff_plan* p) {
  Model md;
  if (!p || check_model(m, &md) != FF_OK || md.L != p->L) return 0;
  if (p->s.feature_mode != FF_RESIDUAL || p->s.mode == FF_VANILLA) return 0;
  try {
    return plan_runs(*p).size() * (size_t)p->s.S * md.E() * sizeof(float);
  } catch (...) {
    return 0;
  }
}

ff_status ff_ctx_hist_sums(ff_ctx* c, void* buf, size_t bytes) {
  try {
    if (!c) return fail(FF_E_NULL, "ctx is NULL");
    if (!buf) {
      c->hsum = nullptr;
      c->runs.clear();
      return ok();
    }
    const ff_plan& p = c->plan;
    if (p.s.feature_mode != FF_RESIDUAL || p.s.mode == FF_VANILLA)
      return fail(FF_E_UNSUPPORTED, "history sums need residual features and a cached mode");
    if (c->next_step != 0) return fail(FF_E_STATE, "history sums are enabled before step 0 (or after ff_ctx_reset)");
    std::vector<std::pair<int, int>> runs = plan_runs(p);
    if (runs.empty()) return fail(FF_E_UNSUPPORTED, "the plan has no run of two or more drafted layers");
    const size_t need = runs.size() * (size_t)p.s.S * c->m.E() * sizeof(float);
    if (bytes < need) return fail(FF_E_WORKSPACE, "history sum buffer %zu < %zu bytes", bytes, need);
    if (!aligned16(buf)) return fail(FF_E_SHAPE, "history sum buffer must be 16-byte aligned");
    c->runs = std::move(runs);
    c->hsum = static_cast<float*>(buf);
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

size_t ff_cond_cache_bytes(const ff_model_desc* m, const ff_plan* p) {
  Model md;
  if (!p || check_model(m, &md) != FF_OK || md.L != p->L) return 0;
  try {
    return cond_layout(md, *p).total;
  } catch (...) {
    return 0;
  }
}

ff_status ff_ctx_cond_cache(ff_ctx* c, void* buf, size_t bytes) {
  try {
    if (!c) return fail(FF_E_NULL, "ctx is NULL");
    if (!buf) {
      c->cc = nullptr;
      c->cc_cond = nullptr;
      return ok();
    }
    if (c->next_step != 0)
      return fail(FF_E_STATE, "the conditioning cache is enabled before step 0 (or after ff_ctx_reset)");
    CondLayout cl = cond_layout(c->m, c->plan);
    if (bytes < cl.total) return fail(FF_E_WORKSPACE, "conditioning cache %zu < %zu bytes", bytes, cl.total);
    if ((uintptr_t)buf % kAlign) return fail(FF_E_SHAPE, "conditioning cache must be %zu-byte aligned", (size_t)kAlign);
    c->cc_lay = std::move(cl);
    c->cc = static_cast<char*>(buf);
    c->cc_cond = nullptr;
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

ff_status ff_ctx_trace(ff_ctx* c, void* buf, size_t bytes) {
  if (!c) return fail(FF_E_NULL, "ctx is NULL");
  if (buf) {
    const size_t need = (size_t)c->m.L * c->m.E() * c->m.es();
    if (bytes < need) return fail(FF_E_WORKSPACE, "trace buffer %zu < %zu bytes", bytes, need);
    if (!aligned16(buf)) return fail(FF_E_SHAPE, "trace buffer must be 16-byte aligned");
  }
  c->trace = buf;
  return ok();
}

ff_status ff_rel_l1(const ff_model_desc* m, const void* a, const void* b, float eps, float* rel, void* ws,
                    size_t ws_bytes, ff_stream_t stream) {
  try {
    Model md;
    ff_status e = check_model(m, &md);
    if (e) return e;
    if (!a || !b || !rel || !ws) return fail(FF_E_NULL, "a, b, rel or ws is NULL");
    if (!(eps > 0.f)) return fail(FF_E_RANGE, "eps must be > 0");
    const Ws L = ws_layout(md);
    if (ws_bytes < L.total) return fail(FF_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);
    if (!aligned16(a) || !aligned16(b) || !aligned16(rel) || !aligned16(ws))
      return fail(FF_E_SHAPE, "pointers must be 16-byte aligned");
    HIP_TRY(ff::rel_l1(md.dtype, a, b, md.B, (size_t)md.N * md.C, eps, rel, at<float>(ws, L.PART),
                       reinterpret_cast<hipStream_t>(stream)), "rel_l1");
    return ok();
  } catch (...) {
    return fail(FF_E_UNSUPPORTED, "unexpected host exception");
  }
}

ff_status ff_ctx_profile(ff_ctx* c, int32_t enable) {
  if (!c) return fail(FF_E_NULL, "ctx is NULL");
  c->prof.on = enable != 0;
  c->prof.recs.clear();
  c->prof.next = 0;
  return ok();
}

ff_status ff_ctx_profile_read(ff_ctx* c, ff_prof_stat* out) {
  if (!c || !out) return fail(FF_E_NULL, "ctx or out is NULL");
  for (int k = 0; k < FF_PROF_NCLASS; ++k) out[k] = ff_prof_stat{0, 0.0, 0.0, 0.0};
  for (const Prof::Rec& r : c->prof.recs) {
    HIP_TRY(hipEventSynchronize(r.b), "profile: event sync");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b), "profile: elapsed");
    ff_prof_stat& o = out[r.cls];
    o.launches++;
    o.ms += ms;
    o.flops += r.flops;
    o.bytes += r.bytes;
  }
  c->prof.recs.clear();
  c->prof.next = 0;
  return ok();
}

}  // extern "C"
