// HBM-bound kernels of the cached step: feature-history refresh, Taylor draft, and the
// fused verify + replace pass.  Every thread moves 16-byte chunks (8 bf16 or 4 fp32) with
// a grid-stride loop so that consecutive lanes touch consecutive chunks (fully coalesced).
#include "dev_common.h"

namespace ff {

namespace {

constexpr int kThreads = 256;

inline int grid_for(size_t chunks) {
  size_t g = (chunks + kThreads - 1) / kThreads;
  if (g > 8192) g = 8192;
  if (g < 1) g = 1;
  return (int)g;
}

// History refresh (Eq. 2 is estimated from exact refreshes): Delta = h - u, or h itself.
template <int DT, bool RES>
__global__ __launch_bounds__(kThreads) void k_cache_update(void* __restrict__ slot, const void* __restrict__ u,
                                                           const void* __restrict__ h, size_t nchunk) {
  using S = St<DT>;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    const size_t i = c * S::V;
    float hv[S::V];
    S::load(h, i, hv);
    if (RES) {
      float uv[S::V];
      S::load(u, i, uv);
#pragma unroll
      for (int j = 0; j < S::V; ++j) hv[j] = hv[j] - uv[j];
    }
    S::store(slot, i, hv);
  }
}

// One chunk of the draft h_d = u + sum_m c_m * slot_m (Eq. 2 in coefficient form) from the
// incoming values uv (ignored without RES), fp32 sums with explicit fma in a fixed order,
// then one rounding to the storage type.  Every draft path (single layer, fused run,
// verify) goes through this function, so they produce identical bits.
template <int DT, bool RES>
__device__ __forceinline__ void draft_math(const Terms& t, size_t off, const float* uv, float* out) {
  using S = St<DT>;
  float f[S::V];
#pragma unroll
  for (int j = 0; j < S::V; ++j) f[j] = 0.0f;
#pragma unroll
  for (int m = 0; m < kMaxTerms; ++m) {
    if (m < t.n) {
      float s[S::V];
      S::load_nt(t.slot[m], off, s);   // each history value is read once per step
#pragma unroll
      for (int j = 0; j < S::V; ++j) f[j] = fmaf(t.c[m], s[j], f[j]);
    }
  }
  if (RES) {
#pragma unroll
    for (int j = 0; j < S::V; ++j) f[j] = uv[j] + f[j];
  }
#pragma unroll
  for (int j = 0; j < S::V; ++j) out[j] = S::rnd(f[j]);
}

template <int DT, bool RES>
__device__ __forceinline__ void draft_chunk(const Terms& t, const void* u, size_t i, float* out) {
  using S = St<DT>;
  float uv[S::V];
  if (RES) S::load(u, i, uv);
  draft_math<DT, RES>(t, i, uv, out);
}

template <int DT, bool RES>
__global__ __launch_bounds__(kThreads) void k_draft_run(Terms t, int layers, size_t layer_stride, void* x,
                                                        size_t nchunk) {
  using S = St<DT>;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    const size_t i = c * S::V;
    float xv[S::V];
    if (RES) S::load(x, i, xv);
    // four layers per pass: their history loads do not depend on the running value, so
    // all of them are in flight together
    int l = 0;
    for (; l + 4 <= layers; l += 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q) draft_math<DT, RES>(t, (size_t)(l + q) * layer_stride + i, xv, xv);
    }
    for (; l < layers; ++l) draft_math<DT, RES>(t, (size_t)l * layer_stride + i, xv, xv);
    S::store(x, i, xv);
  }
}

// History sum of a run of drafted layers (residual features): P = sum over the run's
// layers, in layer order, of one ring slot, in fp32.  Eq. 2's draft is linear in the
// history, so a run l0..l1-1 of drafted layers moves the stream by sum_m c_m P_m (P_m the
// sum of slot m over the run): formed once when a refresh rewrites the slot and read by
// every cached step until the slot is rewritten again.
template <int DT>
__global__ __launch_bounds__(kThreads) void k_hist_sum(const void* __restrict__ slot0, int layers, size_t layer_stride,
                                                       float* __restrict__ out, size_t nchunk) {
  using S = St<DT>;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    const size_t i = c * S::V;
    float acc[S::V], v[S::V];
    S::load_nt(slot0, i, acc);
    for (int l = 1; l < layers; ++l) {
      S::load_nt(slot0, (size_t)l * layer_stride + i, v);
#pragma unroll
      for (int j = 0; j < S::V; ++j) acc[j] += v[j];
    }
#pragma unroll
    for (int j = 0; j < S::V; j += 4)
      *reinterpret_cast<float4*>(out + i + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
  }
}

// A whole run of drafted layers from its history sums: x <- round(x + sum_m c_m P_m), the
// terms in fp32 (t.slot[m] points at fp32 sums), one rounding to the storage type.
template <int DT>
__global__ __launch_bounds__(kThreads) void k_draft_sum(Terms t, void* x, size_t nchunk) {
  using S = St<DT>;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    const size_t i = c * S::V;
    float xv[S::V], f[S::V];
    S::load(x, i, xv);
#pragma unroll
    for (int j = 0; j < S::V; ++j) f[j] = 0.0f;
#pragma unroll
    for (int m = 0; m < kMaxTerms; ++m) {
      if (m < t.n) {
#pragma unroll
        for (int j = 0; j < S::V; j += 4) {
          float p[4];
          St<DT_F32>::load_nt(t.slot[m], i + j, p);
#pragma unroll
          for (int q = 0; q < 4; ++q) f[j + q] = fmaf(t.c[m], p[q], f[j + q]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < S::V; ++j) xv[j] = S::rnd(xv[j] + f[j]);
    S::store(x, i, xv);
  }
}

template <int DT, bool RES>
__global__ __launch_bounds__(kThreads) void k_draft(Terms t, const void* u, void* hd, size_t nchunk) {
  using S = St<DT>;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    float o[S::V];
    draft_chunk<DT, RES>(t, u, c * S::V, o);
    S::store(hd, c * S::V, o);
  }
}

// Block-wide fixed-order sum of two values (wave butterflies, then waves in order).
__device__ __forceinline__ void block_sum2(float& a, float& b) {
  __shared__ float red[2][kThreads / 64];
  a = wave_sum(a);
  b = wave_sum(b);
  const int w = threadIdx.x / 64, l = threadIdx.x % 64;
  if (l == 0) { red[0][w] = a; red[1][w] = b; }
  __syncthreads();
  if (threadIdx.x == 0) {
    float x = 0.f, y = 0.f;
#pragma unroll
    for (int i = 0; i < kThreads / 64; ++i) { x += red[0][i]; y += red[1][i]; }
    a = x; b = y;
  }
}

constexpr int kMaxVerifyBlocks = 2048;  // partial-sum blocks per sample

// Verify + replace (Eq. 3-5): rebuild the draft from the same incoming u, accumulate
// sum|h_d - h_f| and sum|h_f| for this sample, and forward h_f (FeatFix) or h_d (Verify).
template <int DT, bool RES>
__global__ __launch_bounds__(kThreads) void k_verify(Terms t, const void* u, const void* __restrict__ hf,
                                                     void* hout, Forward fw, size_t chunks_per_sample,
                                                     float* __restrict__ partials) {
  using S = St<DT>;
  const int b = blockIdx.y;
  const size_t base = (size_t)b * chunks_per_sample * S::V;
  float num = 0.f, den = 0.f;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < chunks_per_sample;
       c += (size_t)gridDim.x * kThreads) {
    const size_t i = base + c * S::V;
    float d[S::V], f[S::V];
    draft_chunk<DT, RES>(t, u, i, d);
    S::load(hf, i, f);
#pragma unroll
    for (int j = 0; j < S::V; ++j) {
      num += fabsf(d[j] - f[j]);
      den += fabsf(f[j]);
    }
    if (fw.kind == FWD_DRAFT || fw.kind == FWD_EXACT) {
      S::store(hout, i, fw.kind == FWD_EXACT ? f : d);
    } else {
      // partial forwarding: a chunk lies in one row (C % V == 0); row n = e / C, channel e % C
      const size_t e = c * S::V;
      const int n = (int)(e / fw.C), ch = (int)(e % fw.C);
      float o[S::V];
#pragma unroll
      for (int j = 0; j < S::V; ++j) {
        const bool exact = fw.kind == FWD_TOKENS ? n % fw.stride == 0 : (ch + j) % fw.stride == 0;
        o[j] = exact ? f[j] : d[j];
      }
      S::store(hout, i, o);
    }
  }
  block_sum2(num, den);
  if (threadIdx.x == 0) {
    float* p = partials + ((size_t)b * gridDim.x + blockIdx.x) * 2;
    p[0] = num;
    p[1] = den;
  }
}

// First stage of the rel-L1 distance of two tensors (the audit's reduction without a
// draft): per block, sum |a - b| and |b| over its share of one sample.
template <int DT>
__global__ __launch_bounds__(kThreads) void k_rel_partials(const void* __restrict__ a, const void* __restrict__ b,
                                                           size_t chunks_per_sample, float* __restrict__ partials) {
  using S = St<DT>;
  const int smp = blockIdx.y;
  const size_t base = (size_t)smp * chunks_per_sample * S::V;
  float num = 0.f, den = 0.f;
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < chunks_per_sample;
       c += (size_t)gridDim.x * kThreads) {
    float x[S::V], y[S::V];
    S::load(a, base + c * S::V, x);
    S::load(b, base + c * S::V, y);
#pragma unroll
    for (int j = 0; j < S::V; ++j) {
      num += fabsf(x[j] - y[j]);
      den += fabsf(y[j]);
    }
  }
  block_sum2(num, den);
  if (threadIdx.x == 0) {
    float* p = partials + ((size_t)smp * gridDim.x + blockIdx.x) * 2;
    p[0] = num;
    p[1] = den;
  }
}

// Second stage: per sample, sum the partials in index order and form Eq. 4.
__global__ __launch_bounds__(kThreads) void k_verify_finish(const float* __restrict__ partials, int nblk,
                                                            float eps, float* __restrict__ rel) {
  const int b = blockIdx.x;
  float num = 0.f, den = 0.f;
  for (int i = threadIdx.x; i < nblk; i += kThreads) {
    num += partials[((size_t)b * nblk + i) * 2];
    den += partials[((size_t)b * nblk + i) * 2 + 1];
  }
  block_sum2(num, den);
  if (threadIdx.x == 0) rel[b] = num / (den + eps);
}

template <int DT>
__global__ __launch_bounds__(kThreads) void k_copy_rows(const void* __restrict__ src, void* __restrict__ dst,
                                                        int n, int N, int off, int C, size_t nchunk) {
  using S = St<DT>;
  const int cpr = C / S::V;  // chunks per row
  for (size_t c = (size_t)blockIdx.x * kThreads + threadIdx.x; c < nchunk; c += (size_t)gridDim.x * kThreads) {
    const size_t row = c / cpr;
    const int col = (int)(c % cpr) * S::V;
    const size_t b = row / n, i = row % n;
    float v[S::V];
    S::load(src, row * C + col, v);
    S::store(dst, (b * N + off + i) * C + col, v);
  }
}

}  // namespace

hipError_t cache_update(int dtype, void* slot, const void* u, const void* h, size_t E, hipStream_t s) {
  if (dtype == DT_BF16) {
    size_t n = E / 8;
    if (u) FF_LAUNCH((k_cache_update<DT_BF16, true>), grid_for(n), kThreads, 0, s, slot, u, h, n);
    else FF_LAUNCH((k_cache_update<DT_BF16, false>), grid_for(n), kThreads, 0, s, slot, u, h, n);
  } else {
    size_t n = E / 4;
    if (u) FF_LAUNCH((k_cache_update<DT_F32, true>), grid_for(n), kThreads, 0, s, slot, u, h, n);
    else FF_LAUNCH((k_cache_update<DT_F32, false>), grid_for(n), kThreads, 0, s, slot, u, h, n);
  }
  return hipGetLastError();
}

hipError_t draft(int dtype, const Terms& t, const void* u, void* hd, size_t E, hipStream_t s) {
  if (dtype == DT_BF16) {
    size_t n = E / 8;
    if (u) FF_LAUNCH((k_draft<DT_BF16, true>), grid_for(n), kThreads, 0, s, t, u, hd, n);
    else FF_LAUNCH((k_draft<DT_BF16, false>), grid_for(n), kThreads, 0, s, t, u, hd, n);
  } else {
    size_t n = E / 4;
    if (u) FF_LAUNCH((k_draft<DT_F32, true>), grid_for(n), kThreads, 0, s, t, u, hd, n);
    else FF_LAUNCH((k_draft<DT_F32, false>), grid_for(n), kThreads, 0, s, t, u, hd, n);
  }
  return hipGetLastError();
}

hipError_t draft_run(int dtype, const Terms& t, int layers, size_t layer_stride, int residual, void* x, size_t E,
                     hipStream_t s) {
  if (dtype == DT_BF16) {
    size_t n = E / 8;
    if (residual) FF_LAUNCH((k_draft_run<DT_BF16, true>), grid_for(n), kThreads, 0, s, t, layers, layer_stride, x, n);
    else FF_LAUNCH((k_draft_run<DT_BF16, false>), grid_for(n), kThreads, 0, s, t, layers, layer_stride, x, n);
  } else {
    size_t n = E / 4;
    if (residual) FF_LAUNCH((k_draft_run<DT_F32, true>), grid_for(n), kThreads, 0, s, t, layers, layer_stride, x, n);
    else FF_LAUNCH((k_draft_run<DT_F32, false>), grid_for(n), kThreads, 0, s, t, layers, layer_stride, x, n);
  }
  return hipGetLastError();
}

hipError_t hist_sum(int dtype, const void* slot0, int layers, size_t layer_stride, float* out, size_t E,
                    hipStream_t s) {
  if (layers < 1) return hipErrorInvalidValue;
  if (dtype == DT_BF16) {
    const size_t n = E / 8;
    FF_LAUNCH((k_hist_sum<DT_BF16>), grid_for(n), kThreads, 0, s, slot0, layers, layer_stride, out, n);
  } else {
    const size_t n = E / 4;
    FF_LAUNCH((k_hist_sum<DT_F32>), grid_for(n), kThreads, 0, s, slot0, layers, layer_stride, out, n);
  }
  return hipGetLastError();
}

hipError_t draft_sum(int dtype, const Terms& t, void* x, size_t E, hipStream_t s) {
  if (t.n < 1 || t.n > kMaxTerms) return hipErrorInvalidValue;
  if (dtype == DT_BF16) FF_LAUNCH((k_draft_sum<DT_BF16>), grid_for(E / 8), kThreads, 0, s, t, x, E / 8);
  else FF_LAUNCH((k_draft_sum<DT_F32>), grid_for(E / 4), kThreads, 0, s, t, x, E / 4);
  return hipGetLastError();
}

size_t verify_partials_floats(int B) { return (size_t)B * kMaxVerifyBlocks * 2; }

hipError_t verify(int dtype, const Terms& t, const void* u, const void* hf, void* hout, const Forward& fw,
                  int B, size_t Eb, float eps, float* rel_l1, float* partials, hipStream_t s) {
  if (fw.kind < FWD_DRAFT || fw.kind > FWD_CHANNELS) return hipErrorInvalidValue;
  if (fw.kind >= FWD_TOKENS && (fw.stride < 1 || fw.C < 1 || fw.C % (dtype == DT_BF16 ? 8 : 4))) return hipErrorInvalidValue;
  const int V = dtype == DT_BF16 ? 8 : 4;
  const size_t cps = Eb / V;
  int nblk = cdiv((long)cps, kThreads);
  if (nblk > kMaxVerifyBlocks) nblk = kMaxVerifyBlocks;
  if (nblk < 1) nblk = 1;
  dim3 grid(nblk, B);
  if (dtype == DT_BF16) {
    if (u) FF_LAUNCH((k_verify<DT_BF16, true>), grid, kThreads, 0, s, t, u, hf, hout, fw, cps, partials);
    else FF_LAUNCH((k_verify<DT_BF16, false>), grid, kThreads, 0, s, t, u, hf, hout, fw, cps, partials);
  } else {
    if (u) FF_LAUNCH((k_verify<DT_F32, true>), grid, kThreads, 0, s, t, u, hf, hout, fw, cps, partials);
    else FF_LAUNCH((k_verify<DT_F32, false>), grid, kThreads, 0, s, t, u, hf, hout, fw, cps, partials);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (rel_l1) FF_LAUNCH(k_verify_finish, dim3(B), kThreads, 0, s, partials, nblk, eps, rel_l1);
  return hipGetLastError();
}

hipError_t rel_l1(int dtype, const void* a, const void* b, int B, size_t Eb, float eps, float* rel, float* partials,
                  hipStream_t s) {
  const int V = dtype == DT_BF16 ? 8 : 4;
  const size_t cps = Eb / V;
  int nblk = cdiv((long)cps, kThreads);
  if (nblk > kMaxVerifyBlocks) nblk = kMaxVerifyBlocks;
  if (nblk < 1) nblk = 1;
  if (dtype == DT_BF16) FF_LAUNCH(k_rel_partials<DT_BF16>, dim3(nblk, B), kThreads, 0, s, a, b, cps, partials);
  else FF_LAUNCH(k_rel_partials<DT_F32>, dim3(nblk, B), kThreads, 0, s, a, b, cps, partials);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  FF_LAUNCH(k_verify_finish, dim3(B), kThreads, 0, s, partials, nblk, eps, rel);
  return hipGetLastError();
}

hipError_t copy_rows(int dtype, const void* src, void* dst, int B, int n, int N, int off, int C, hipStream_t st) {
  const int V = dtype == DT_BF16 ? 8 : 4;
  size_t nchunk = (size_t)B * n * (C / V);
  if (nchunk == 0) return hipSuccess;
  if (dtype == DT_BF16) FF_LAUNCH(k_copy_rows<DT_BF16>, grid_for(nchunk), kThreads, 0, st, src, dst, n, N, off, C, nchunk);
  else FF_LAUNCH(k_copy_rows<DT_F32>, grid_for(nchunk), kThreads, 0, st, src, dst, n, N, off, C, nchunk);
  return hipGetLastError();
}

}  // namespace ff
