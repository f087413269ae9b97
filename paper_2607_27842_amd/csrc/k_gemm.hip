// Dense contractions of the exact block: out = epi(A W^T + bias) with A [M, K] (rows
// through a RowMap), W [N, K] (both K-contiguous), fp32 accumulation.
//
// bf16: v_mfma_f32_16x16x32_bf16 on 256x256 or 128x128 workgroup tiles; operands staged
// through LDS (row stride padded by 16 bytes so that the 16-byte fragment reads of 16
// consecutive rows are conflict-free), double-buffered with one barrier per K step; the
// next K step's global loads are in flight while the current one is multiplied.
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

// Epilogue for 4 consecutive output columns c..c+3 of row r (N % 8 == 0, so all four are
// in range when c is): 8/16-byte loads of bias, gate and residual and one vector store.
template <int EPI, bool OUT_F32, bool RES_F32>
__device__ __forceinline__ void epilogue4_bf16(const GemmArgs a, int r, int c, f32x4_t acc) {
  const uint16_t* bias = reinterpret_cast<const uint16_t*>(a.bias);
  const u32x2_t bw = *reinterpret_cast<const u32x2_t*>(bias + c);
  float v[4] = {acc[0] + __uint_as_float(bw[0] << 16), acc[1] + __uint_as_float(bw[0] & 0xffff0000u),
                acc[2] + __uint_as_float(bw[1] << 16), acc[3] + __uint_as_float(bw[1] & 0xffff0000u)};
  if (EPI == EPI_BIAS_GELU) {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = gelu_tanh_f(v[j]);
  }
  const size_t pr = (size_t)a.omap.phys(r);
  if (EPI == EPI_GATED) {
    float res[4];
    if (RES_F32) {
      const f32x4_t q = *reinterpret_cast<const f32x4_t*>(reinterpret_cast<const float*>(a.resid) + pr * a.ldr + c);
      res[0] = q[0]; res[1] = q[1]; res[2] = q[2]; res[3] = q[3];
    } else {
      const u32x2_t q = *reinterpret_cast<const u32x2_t*>(reinterpret_cast<const uint16_t*>(a.resid) + pr * a.ldr + c);
      res[0] = __uint_as_float(q[0] << 16); res[1] = __uint_as_float(q[0] & 0xffff0000u);
      res[2] = __uint_as_float(q[1] << 16); res[3] = __uint_as_float(q[1] & 0xffff0000u);
    }
    const f32x4_t g = *reinterpret_cast<const f32x4_t*>(a.gate + (size_t)a.omap.sample(r) * a.ldg + c);
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = res[j] + g[j] * v[j];
  }
  if (OUT_F32) {
    const f32x4_t o = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4_t*>(reinterpret_cast<float*>(a.out) + pr * a.ldo + c) = o;
  } else {
    u32x2_t o;
    o[0] = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
    o[1] = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
    *reinterpret_cast<u32x2_t*>(reinterpret_cast<uint16_t*>(a.out) + pr * a.ldo + c) = o;
  }
}

// Workgroup -> output tile.  Workgroups are dispatched round-robin over the 8 XCDs (each
// with its own L2); the first floor(n/8)*8 of them are renumbered so that every XCD owns
// a contiguous range of tiles, and tiles are ordered in groups of kGroupM tile-rows so
// that an XCD's concurrent tiles share A rows and W columns in its L2.
constexpr int kGroupM = 8;
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  const int full = (nwg / 8) * 8;
  const int id = bid < full ? (bid % 8) * (full / 8) + bid / 8 : bid;
  const int per_group = kGroupM * tiles_n;
  const int first_m = (id / per_group) * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in_group = id % per_group;
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
// BM x BN workgroup tile, BK = 64, wavefront tiles WM x WN of 16x16x32 MFMAs.  The MFMA
// takes the weight fragment as its A operand and the activation fragment as B, so the
// accumulator of a lane holds 4 consecutive output COLUMNS of one output row: the fused
// epilogue reads bias / gate / residual and writes the result with vector accesses.
constexpr int BK = 64, LDT = BK + 8;

template <int BM, int BN, int WM, int WN, int EPI, bool OUT_F32, bool RES_F32>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void k_gemm_bf16(GemmArgs a, int tiles_m, int tiles_n) {
  constexpr int NWN = BN / WN;
  constexpr int NT = (BM / WM) * NWN * 64;
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int RSTEP = NT / 8;            // rows covered by one pass of 16-byte chunk loads
  constexpr int CA = BM / RSTEP, CB = BN / RSTEP;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(a.A);
  const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);

  const int lrow = tid >> 3, kc = (tid & 7) * 8;
  size_t offa[CA], offb[CB];
  unsigned mask = 0;
#pragma unroll
  for (int i = 0; i < CA; ++i) {
    const int gm = m0 + lrow + RSTEP * i;
    if (gm < a.M) mask |= 1u << i;
    offa[i] = (size_t)(gm < a.M ? a.amap.phys(gm) : 0) * a.lda + kc;
  }
#pragma unroll
  for (int i = 0; i < CB; ++i) {
    const int gn = n0 + lrow + RSTEP * i;
    if (gn < a.N) mask |= 1u << (16 + i);
    offb[i] = (size_t)(gn < a.N ? gn : 0) * a.ldw + kc;
  }
  u32x4_t ra[CA], rb[CB];
  const u32x4_t z4 = {0u, 0u, 0u, 0u};
#define FF_GLOAD(k0)                                                                                   \
  do {                                                                                                 \
    const bool kin = (k0) + kc < a.K;                                                                  \
    _Pragma("unroll") for (int i = 0; i < CA; ++i)                                                     \
      ra[i] = (kin && (mask & (1u << i))) ? *reinterpret_cast<const u32x4_t*>(A + offa[i] + (k0)) : z4; \
    _Pragma("unroll") for (int i = 0; i < CB; ++i)                                                     \
      rb[i] = (kin && (mask & (1u << (16 + i)))) ? *reinterpret_cast<const u32x4_t*>(W + offb[i] + (k0)) : z4; \
  } while (0)
#define FF_SSTORE(buf)                                                                                 \
  do {                                                                                                 \
    _Pragma("unroll") for (int i = 0; i < CA; ++i)                                                     \
      *reinterpret_cast<u32x4_t*>(&sA[buf][(lrow + RSTEP * i) * LDT + kc]) = ra[i];                    \
    _Pragma("unroll") for (int i = 0; i < CB; ++i)                                                     \
      *reinterpret_cast<u32x4_t*>(&sB[buf][(lrow + RSTEP * i) * LDT + kc]) = rb[i];                    \
  } while (0)

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int wm = (wave / NWN) * WM, wn = (wave % NWN) * WN;
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
      bf16x8_t fa[TM], fb[TN];
#pragma unroll
      for (int t = 0; t < TM; ++t)
        fa[t] = *reinterpret_cast<const bf16x8_t*>(&sA[cur][(wm + t * 16 + fr) * LDT + kk + fk]);
#pragma unroll
      for (int t = 0; t < TN; ++t)
        fb[t] = *reinterpret_cast<const bf16x8_t*>(&sB[cur][(wn + t * 16 + fr) * LDT + kk + fk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) FF_SSTORE(cur ^ 1);
    __syncthreads();
  }
#undef FF_GLOAD
#undef FF_SSTORE
  // acc[i][j][v] = C[row m0 + wm + 16i + (lane % 16)][col n0 + wn + 16j + 4*(lane / 16) + v]
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = m0 + wm + i * 16 + fr;
    if (r >= a.M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int c = n0 + wn + j * 16 + (lane >> 4) * 4;
      if (c < a.N) epilogue4_bf16<EPI, OUT_F32, RES_F32>(a, r, c, acc[i][j]);
    }
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

template <int BM, int BN, int WM, int WN, int EPI, bool OF, bool RF>
void launch_tile(const GemmArgs& a, hipStream_t s) {
  const int tm = (a.M + BM - 1) / BM, tn = (a.N + BN - 1) / BN;
  hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, EPI, OF, RF>), tm * tn, (BM / WM) * (BN / WN) * 64, 0, s, a, tm, tn);
}

// 256x256 tiles (8 wavefronts of 128x64, one workgroup per CU) when there are enough of
// them to fill the chip; otherwise 128x128 tiles (4 wavefronts of 64x64, two per CU).
template <int EPI, bool OF, bool RF>
void launch_bf16(const GemmArgs& a, hipStream_t s) {
  const long big = (long)((a.M + 255) / 256) * ((a.N + 255) / 256);
  if (big >= 200) launch_tile<256, 256, 128, 64, EPI, OF, RF>(a, s);
  else launch_tile<128, 128, 64, 64, EPI, OF, RF>(a, s);
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
