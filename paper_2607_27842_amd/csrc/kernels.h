// Internal interface between the host library (featfix.cpp) and the gfx950 kernels.
// Not part of the public ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ff {

enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Events for the next kernel launch (set by the host profiler, consumed and cleared by
// the launch): the kernel is then started with hipExtLaunchKernelGGL, which records
// `start` / `stop` at the kernel's own execution boundaries.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchEvents g_launch_events;
constexpr int kMaxTerms = 4;  // forecast order K <= 3 -> at most 4 history terms

inline size_t dsize(int dt) { return dt == DT_BF16 ? 2 : 4; }

// Logical row r of a stream segment -> physical row of a [B, N, *] tensor:
// sample b = r / n_seg, physical row b * N + off + r % n_seg.  For a whole tensor
// n_seg == N and off == 0 (identity).  MMDiT text rows: (n_txt, N, 0); image rows:
// (n_img, N, n_txt).
struct RowMap {
  int n_seg, N, off;
  __host__ __device__ inline int phys(int r) const { return (r / n_seg) * N + off + r % n_seg; }
  __host__ __device__ inline int sample(int r) const { return r / n_seg; }
};

// ---------------------------------------------------------------- GEMM  (dense contraction)
// out[phys(r), n] = epi( sum_k A[phys(r), k] * W[n, k] + bias[n] ), r < M, n < N.
enum Epi { EPI_BIAS = 0, EPI_BIAS_GELU = 1, EPI_GATED = 2 };
struct GemmArgs {
  const void* A; int lda; RowMap amap;   // model dtype
  const void* W; int ldw;                // [N, K] model dtype
  const void* bias;                      // [N] model dtype (never NULL)
  int M, N, K;
  int epi;
  void* out; int ldo; RowMap omap; int out_f32;  // output fp32 or model dtype
  // EPI_GATED: out = resid[omap.phys(r), n] + gate[sample(r) * ldg + n] * (acc + bias[n])
  const void* resid; int ldr; int resid_f32;
  const float* gate; int ldg;
  // bf16 EPI_GATED with a bf16 output only: also refresh a history slot laid out like out,
  // cache_out[phys(r), n] = round(out - cache_u[phys(r), n]) (cache_u == NULL: = out)
  void* cache_out; const void* cache_u;
};
hipError_t gemm(int dtype, const GemmArgs& a, hipStream_t s);
// Two GEMMs in one launch (bf16) when they share out_f32 and resid_f32 and either share epi
// or mix EPI_BIAS with EPI_BIAS_GELU, and when the combined grid does not take more rounds
// over the CUs; otherwise two launches.  Same results as two gemm() calls.
hipError_t gemm2(int dtype, const GemmArgs& a0, const GemmArgs& a1, hipStream_t s);

// y[b, n] = (add ? add[b*ldadd + n] : 0) + act( sum_k f(x[b*ldx + k]) * W[n, k] + bias[n] )
// x, y, add fp32; W, bias model dtype; f = SiLU if silu_in; act = SiLU if silu_out.
// 1 <= B <= kGemvMaxB.  bf16 weights run on MFMA (K % 8 == 0, x 16-byte aligned rows), each
// weight load serving up to four groups of 8 samples: f(x) enters as bf16 hi + lo parts,
// f(x) = hi + lo to ~2^-17, split in the kernel, or read from xs when set ([16 * groups,
// K] bf16: sample b = 8g + r has hi in row 16g + r and lo in row 16g + 8 + r, as silu_rows
// writes it; the caller guarantees it holds the split of this f(x)).  fp32 weights run in
// groups of 8 samples, one launch each.
constexpr int kGemvMaxB = 32;
struct GemvArgs {
  const float* x; int ldx; int silu_in;
  const void* W; const void* bias;
  int Nout, K, B;
  float* y; int ldy; int silu_out;
  const float* add; int ldadd;
  const uint16_t* xs;
};
hipError_t gemv(int dtype, const GemvArgs& a, hipStream_t s);
// Up to kGemvJobs GEMVs sharing x (and K, B, SiLU on input) in one launch; no add term,
// no SiLU on output.  1 <= B <= kGemvMaxB.
constexpr int kGemvJobs = 32;
struct GemvJob {
  const void* W; const void* bias; float* y;
  int Nout, ldy;
};
struct GemvBatch {
  const float* x; int ldx; int silu_in;
  int K, B, njobs;
  const uint16_t* xs;   // as GemvArgs::xs
  GemvJob job[kGemvJobs];
};
inline size_t gemv_xs_bytes(int K) { return (size_t)16 * (kGemvMaxB / 8) * K * 2; }
hipError_t gemv_batch(int dtype, const GemvBatch& bt, hipStream_t s);

// ---------------------------------------------------------------- history / draft terms
// Terms of a draft: sum_m c[m] * slot[m], m < n, in a fixed order (fp32 fmas from zero).
struct Terms {
  int n;                         // k_eff + 1
  const void* slot[kMaxTerms];   // cache slots (model dtype, E elements each) or fp32 history sums
  float c[kMaxTerms];            // forecast coefficients
};

// ---------------------------------------------------------------- normalisation
// out[phys(r), :C] = LN(in[phys(r), :C]) * (1 + scale[b*ldm + :]) + shift[b*ldm + :]
// With pre.n > 0 (input in the model dtype, not in_f32): a run of drafted layers is
// applied to the row first from its fp32 history sums laid out like in,
//   in[phys(r), :] <- round(in + sum_m pre.c[m] * pre.slot[m][phys(r), :])
// exactly as draft_sum computes it, the row is written back to in, and the LayerNorm
// normalises the updated row.
struct LnModArgs {
  const void* in; int in_f32; int ldi;
  RowMap map; int rows, C; float eps;
  const float* shift; const float* scale; int ldm;
  void* out; int ldo;   // model dtype
  Terms pre;
};
hipError_t ln_modulate(int dtype, const LnModArgs& a, hipStream_t s);

// In-place per-head RMSNorm of columns [col0, col0 + H*d) of x (model dtype):
// x_h <- x_h * g / sqrt(mean(x_h^2) + eps) for each row r < rows (physical via map).
struct RmsArgs {
  void* x; int ld; RowMap map; int rows, H, d, col0;
  const void* g; float eps;
};
hipError_t rms_heads(int dtype, const RmsArgs& a, hipStream_t s);
// Rotary embedding applied after the q / k norms: head dims split into chunks of axes[a]
// (all 0: none); the pair (2i, 2i+1) of chunk a turns by pos_a * theta^(-2i / axes[a]),
// pos = (0, 0, 0) for rows n < n_txt of a sample, else (frame, row, column) of image row
// t = n - n_txt in a (., Hp, Wp) patch grid.
struct Rope {
  int axes[3]; float log2_theta;
  int n_txt, Hp, Wp;
};
// Both per-head RMSNorms of a qkv row block: q at columns [0, H*d) with gain gq, k at
// [H*d, 2*H*d) with gain gk (in place), then the rotary embedding of q and k.
struct RmsQKArgs {
  void* x; int ld; RowMap map; int rows, H, d;
  const void* gq; const void* gk; float eps;
  Rope rope;
};
hipError_t rms_qk(int dtype, const RmsQKArgs& a, hipStream_t s);

// ---------------------------------------------------------------- attention
// out[b*N + i, h*d + e] = softmax_j(q_i . k_j * scale) v_j,  q/k/v read from
// qkv[(b*N + j) * ldq + {0, C, 2C} + h*d + e].
struct AttnArgs {
  const void* qkv; int ldq;
  void* out; int ldo;
  int B, N, H, d, C;
  float scale;
};
hipError_t attention(int dtype, const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------- history / draft / verify
// slot = round(h - u) (residual) or h (u == nullptr)
hipError_t cache_update(int dtype, void* slot, const void* u, const void* h, size_t E, hipStream_t s);
// hd = round((u ? u : 0) + sum_m c_m slot_m)
hipError_t draft(int dtype, const Terms& t, const void* u, void* hd, size_t E, hipStream_t s);
// A run of consecutive drafted layers l0..l0+layers-1 applied in one pass: for every
// element, x <- round(x + sum_m c_m slot_{l,m}) (or round(sum_m ...) without u) layer after
// layer in registers.  slot[m] points at layer l0's m-th slot; layer l's is layer_stride
// elements further.  Bit-identical to `layers` draft() calls.
hipError_t draft_run(int dtype, const Terms& t, int layers, size_t layer_stride, int residual, void* x, size_t E,
                     hipStream_t s);
// History sums for runs of drafted layers (residual features): out = sum_{l < layers} of
// the slot at slot0 + l * layer_stride, in layer order, fp32 [E].
hipError_t hist_sum(int dtype, const void* slot0, int layers, size_t layer_stride, float* out, size_t E,
                    hipStream_t s);
// A run applied from its history sums: x <- round(x + sum_m c_m P_m), t.slot[m] = fp32 P_m.
hipError_t draft_sum(int dtype, const Terms& t, void* x, size_t E, hipStream_t s);
// Fused draft rebuild + rel-L1 partial sums + forwarding, then a fixed-order reduction.
// What the pass writes to hout: the draft, the exact output, or the exact output on every
// stride-th row (token) / channel of a sample with C channels and the draft elsewhere.
enum { FWD_DRAFT = 0, FWD_EXACT = 1, FWD_TOKENS = 2, FWD_CHANNELS = 3 };
struct Forward { int kind, stride, C; };
size_t verify_partials_floats(int B);
hipError_t verify(int dtype, const Terms& t, const void* u, const void* hf, void* hout, const Forward& fw,
                  int B, size_t Eb, float eps, float* rel_l1, float* partials, hipStream_t s);
// rel[b] = sum|a - b| / (sum|b| + eps) over sample b's Eb elements (the audit's fixed-order
// two-stage reduction; partials as for verify)
hipError_t rel_l1(int dtype, const void* a, const void* b, int B, size_t Eb, float eps, float* rel, float* partials,
                  hipStream_t s);

// ---------------------------------------------------------------- small per-step kernels
// phi[k] = cos(s f_k), phi[128 + k] = sin(s f_k), f_k = exp(-ln(1e4) k / 128), in fp64.
hipError_t time_embed(double s, float* phi, hipStream_t st);
// The same embedding for every step of a schedule: phi[i * 256 + :] for s_i = 1000 (1 - i / T),
// i < n (the conditioning does not depend on the latent, so all steps can be formed at once).
hipError_t time_embed_steps(double T, int n, float* phi, hipStream_t st);
// SiLU(c_t) of steps i < nsteps and model rows b < B, c_t = cond[b, :] + u[i, :] (fp32).
// xs set (bf16 models): its bf16 hi / lo split in the GemvArgs::xs layout of step i at
// xs + i * 16 * groups * C (groups = ceil(B / 8)); rows of absent samples are zero.
// Otherwise (fp32 models): cs[(i * B + b) * C + :].  zb[0, nzb) is zeroed (a bias of zeros).
hipError_t cond_split(const float* u, const float* cond, int nsteps, int B, int C, uint16_t* xs, float* cs,
                      uint16_t* zb, int nzb, hipStream_t st);
// Modulation vectors from a GEMM over hi / lo split rows: for step blocks j < nb and model
// rows b < B (R16 = 16 * ceil(B / 8) GEMM rows per block, hi row 16 (b/8) + b%8, lo row 8
// further):  dst[(j * B + b) * ldy + n] = (out[hi, n] + out[lo, n]) + bias[n],  n < N.
// out fp32 [nb * R16, N]; bias model dtype; N % 4 == 0.
hipError_t mod_combine(int dtype, const float* out, int N, const void* bias, float* dst, int ldy, int nb, int B,
                       hipStream_t st);
// y[b*n + k] = silu(x[b*n + k]) for k < n; with xs (B <= kGemvMaxB) also its bf16 hi / lo split
// for the MFMA GEMVs (GemvArgs::xs layout, K = n)
hipError_t silu_rows(const float* x, float* y, int B, int n, uint16_t* xs, hipStream_t st);
// patches[(b*n_img + tok), feat] (model dtype) from latent x[B, lat_c, F, H, W] fp32
// B: model rows; lat_B: latent samples (0: B), patch sample b reads latent b % lat_B;
// cfg_half > 0: rows b and b + cfg_half are a conditional / unconditional pair of latent b
// and the Euler update uses v = v_u + cfg_scale * (v_c - v_u)
struct PatchGeom { int B, lat_c, F, H, W, pt, ph, pw; int lat_B = 0, cfg_half = 0; float cfg_scale = 0.f; };
hipError_t patchify(int dtype, const float* x, void* patches, const PatchGeom& g, hipStream_t st);
// x[b, ch, f, y, x] += dt * yv[(b*n_img + tok), feat], feat order (dt, dy, dx, ch), for the
// latent samples b (guided as PatchGeom says)
hipError_t unpatchify_euler(const float* yv, float* x, float dt, const PatchGeom& g, hipStream_t st);
// Fused final layer of the image rows + unpatchify + Euler, one wavefront per token:
// a = round(LN(in[phys(r)]) (1 + scale[b]) + shift[b]) (model dtype, as ln_modulate),
// v = a W^T + bias (fp32, P = pt*ph*pw*lat_c outputs, W [P, C] model dtype), then
// x[pixel of (r, o)] += dt * v[o] with feature order (dt, dy, dx, ch) as unpatchify_euler.
// The same values as ln_modulate -> gemm (fp32 out) -> unpatchify_euler up to fp32
// summation order.  Every wavefront reads the whole final weight from the caches, so this
// pays only for small weights: final_layer_ok(dtype, P, C); the caller uses the three-
// kernel path otherwise (there a GEMM reuses the weight across its tiles).
struct FinalArgs {
  const void* in; int ldi; RowMap map; int rows, C; float eps;
  const float* shift; const float* scale; int ldm;
  const void* W; const void* bias;
  float* x; float dt; PatchGeom g;
};
bool final_layer_ok(int dtype, int P, int C);
hipError_t final_layer(int dtype, const FinalArgs& a, hipStream_t st);
// dst[(b*N + off + i) * C + :] = src[(b*n + i) * C + :]  (model dtype rows)
hipError_t copy_rows(int dtype, const void* src, void* dst, int B, int n, int N, int off, int C, hipStream_t st);

}  // namespace ff
