// Dense contractions of the exact block: out = epi(A W^T + bias) with A [M, K] (rows
// through a RowMap), W [N, K] (both K-contiguous), fp32 accumulation.
//
// bf16: 128x128x64 workgroup tile, 4 wavefronts each owning a 64x64 quadrant computed as
// 4x4 v_mfma_f32_16x16x32_bf16 tiles; operands staged through LDS (row stride padded by
// 16 bytes so that the 16-byte fragment reads of 16 consecutive rows are conflict-free),
// double-buffered with one barrier per K step; the next K step's global loads are in
// flight while the current one is multiplied.
// fp32: 64x64x16 tile of plain FMAs (the small fp32 workload is launch-bound).
#include "dev_common.h"

namespace ff {

namespace {

template <int EPI, bool OUT_F32, bool RES_F32, int DT>
__device__ __forceinline__ void epilogue_store(const GemmArgs a, int r, int c, float acc) {
  float v = acc + St<DT>::ld1(a.bias, c);
  if (EPI == EPI_BIAS_GELU) v = gelu_tanh_f(v);
  const size_t pr = (size_t)a.omap.phys(r);
  if (EPI == EPI_GATED) {
    const float res = RES_F32 ? reinterpret_cast<const float*>(a.resid)[pr * a.ldr + c]
                              : St<DT>::ld1(a.resid, pr * a.ldr + c);
    const float g = a.gate[(size_t)a.omap.sample(r) * a.ldg + c];
    v = res + g * v;
  }
  if (OUT_F32) reinterpret_cast<float*>(a.out)[pr * a.ldo + c] = v;
  else St<DT>::st1(a.out, pr * a.ldo + c, v);
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
constexpr int BM = 128, BN = 128, BK = 64, LDT = BK + 8;

template <int EPI, bool OUT_F32, bool RES_F32>
__global__ __launch_bounds__(256) void k_gemm_bf16(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int m0 = (blockIdx.x / tiles_n) * BM, n0 = (blockIdx.x % tiles_n) * BN;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(a.A);
  const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);

  // Global->LDS mapping: 1024 16-byte chunks per operand tile, 4 per thread (rows
  // lrow + 32*i).  Out-of-range rows read row 0 and are zeroed by the mask bits.
  const int lrow = tid >> 3, kc = (tid & 7) * 8;
  size_t offa[4], offb[4];
  unsigned mask = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int gm = m0 + lrow + 32 * i, gn = n0 + lrow + 32 * i;
    if (gm < a.M) mask |= 1u << i;
    if (gn < a.N) mask |= 16u << i;
    offa[i] = (size_t)(gm < a.M ? a.amap.phys(gm) : 0) * a.lda + kc;
    offb[i] = (size_t)(gn < a.N ? gn : 0) * a.ldw + kc;
  }
  u32x4_t ra[4], rb[4];
  const u32x4_t z4 = {0u, 0u, 0u, 0u};
#define FF_GLOAD(k0)                                                                      \
  do {                                                                                    \
    const bool kin = (k0) + kc < a.K;                                                     \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                       \
      ra[i] = (kin && (mask & (1u << i))) ? *reinterpret_cast<const u32x4_t*>(A + offa[i] + (k0)) : z4; \
      rb[i] = (kin && (mask & (16u << i))) ? *reinterpret_cast<const u32x4_t*>(W + offb[i] + (k0)) : z4; \
    }                                                                                     \
  } while (0)
#define FF_SSTORE(buf)                                                                    \
  do {                                                                                    \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                       \
      *reinterpret_cast<u32x4_t*>(&sA[buf][(lrow + 32 * i) * LDT + kc]) = ra[i];            \
      *reinterpret_cast<u32x4_t*>(&sB[buf][(lrow + 32 * i) * LDT + kc]) = rb[i];            \
    }                                                                                     \
  } while (0)

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  const int nk = (a.K + BK - 1) / BK;
  FF_GLOAD(0);
  FF_SSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) FF_GLOAD((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      bf16x8_t fa[4], fb[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        fa[t] = *reinterpret_cast<const bf16x8_t*>(&sA[cur][(wm + t * 16 + fr) * LDT + kk + fk]);
        fb[t] = *reinterpret_cast<const bf16x8_t*>(&sB[cur][(wn + t * 16 + fr) * LDT + kk + fk]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) FF_SSTORE(cur ^ 1);
    __syncthreads();
  }
#undef FF_GLOAD
#undef FF_SSTORE
  // 16x16 accumulator layout: lane holds rows 4*(lane/16) + v, column lane % 16.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int r = m0 + wm + i * 16 + (lane >> 4) * 4 + v;
        const int c = n0 + wn + j * 16 + fr;
        if (r < a.M && c < a.N) epilogue_store<EPI, OUT_F32, RES_F32, DT_BF16>(a, r, c, acc[i][j][v]);
      }
}

// ------------------------------------------------------------------ fp32 FMA GEMM
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs a) {
  constexpr int TM = 64, TN = 64, TK = 16;
  __shared__ __attribute__((aligned(16))) float sA[TK][TM + 4];
  __shared__ __attribute__((aligned(16))) float sB[TK][TN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int tiles_n = (a.N + TN - 1) / TN;
  const int m0 = (blockIdx.x / tiles_n) * TM, n0 = (blockIdx.x % tiles_n) * TN;
  const float* A = reinterpret_cast<const float*>(a.A);
  const float* W = reinterpret_cast<const float*>(a.W);
  const int lrow = tid >> 2, kc = (tid & 3) * 4;
  const bool oka = m0 + lrow < a.M, okb = n0 + lrow < a.N;
  const float* pa = A + (size_t)(oka ? a.amap.phys(m0 + lrow) : 0) * a.lda + kc;
  const float* pb = W + (size_t)(okb ? n0 + lrow : 0) * a.ldw + kc;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += TK) {
    const bool kin = k0 + kc < a.K;
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 va = (oka && kin) ? *reinterpret_cast<const float4*>(pa + k0) : z;
    const float4 vb = (okb && kin) ? *reinterpret_cast<const float4*>(pb + k0) : z;
    __syncthreads();
    sA[kc + 0][lrow] = va.x; sA[kc + 1][lrow] = va.y; sA[kc + 2][lrow] = va.z; sA[kc + 3][lrow] = va.w;
    sB[kc + 0][lrow] = vb.x; sB[kc + 1][lrow] = vb.y; sB[kc + 2][lrow] = vb.z; sB[kc + 3][lrow] = vb.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      const float4 x = *reinterpret_cast<const float4*>(&sA[k][ty * 4]);
      const float4 y = *reinterpret_cast<const float4*>(&sB[k][tx * 4]);
      const float xa[4] = {x.x, x.y, x.z, x.w}, yb[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(xa[i], yb[j], acc[i][j]);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = m0 + ty * 4 + i, c = n0 + tx * 4 + j;
      if (r < a.M && c < a.N) epilogue_store<EPI, true, true, DT_F32>(a, r, c, acc[i][j]);
    }
}

template <int EPI, bool OF, bool RF>
void launch_bf16(const GemmArgs& a, hipStream_t s) {
  const int grid = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((k_gemm_bf16<EPI, OF, RF>), grid, 256, 0, s, a);
}

}  // namespace

hipError_t gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (dtype == DT_F32) {
    const int grid = ((a.M + 63) / 64) * ((a.N + 63) / 64);
    switch (a.epi) {
      case EPI_BIAS: hipLaunchKernelGGL(k_gemm_f32<EPI_BIAS>, grid, 256, 0, s, a); break;
      case EPI_BIAS_GELU: hipLaunchKernelGGL(k_gemm_f32<EPI_BIAS_GELU>, grid, 256, 0, s, a); break;
      default: hipLaunchKernelGGL(k_gemm_f32<EPI_GATED>, grid, 256, 0, s, a); break;
    }
    return hipGetLastError();
  }
  const bool of = a.out_f32 != 0, rf = a.resid_f32 != 0;
  switch (a.epi) {
    case EPI_BIAS:
      if (of) launch_bf16<EPI_BIAS, true, false>(a, s);
      else launch_bf16<EPI_BIAS, false, false>(a, s);
      break;
    case EPI_BIAS_GELU:
      if (of) launch_bf16<EPI_BIAS_GELU, true, false>(a, s);
      else launch_bf16<EPI_BIAS_GELU, false, false>(a, s);
      break;
    default:
      if (of && rf) launch_bf16<EPI_GATED, true, true>(a, s);
      else if (of) launch_bf16<EPI_GATED, true, false>(a, s);
      else if (rf) launch_bf16<EPI_GATED, false, true>(a, s);
      else launch_bf16<EPI_GATED, false, false>(a, s);
      break;
  }
  return hipGetLastError();
}

}  // namespace ff
