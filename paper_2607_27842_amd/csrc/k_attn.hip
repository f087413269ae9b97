// Softmax attention softmax(q k^T * scale) v per (sample, head), flash-style: key/value
// tiles are staged through LDS and each wavefront keeps a running (max, sum) per query
// (online softmax), so no N x N matrix is ever stored.
//
// bf16 (MFMA): a wavefront owns 32 queries (two 16-query groups); a workgroup of 4
// wavefronts shares each 64-key tile.  Scores are formed transposed, S^T = K Q^T, with
// v_mfma_f32_16x16x32_bf16 so that every lane ends up holding the scores of ONE query
// column for 4 keys per 16-key tile: the softmax statistics need only lane-local work
// plus two cross-lane steps, and the probabilities are already in the register layout
// of the B operand of O^T = V^T P^T (no shuffle).  V is transposed into LDS while it is
// staged so that the A operand of that product is two 8-byte LDS reads.  The head dim
// is zero-padded to a multiple of 32 for QK^T and of 16 for PV (d = 72 -> 96 / 80).
// fp32: one thread per query, 32-key LDS tiles (small fp32 workloads only).
#include "dev_common.h"

namespace ff {

namespace {

constexpr int KT = 64;  // keys per LDS tile

template <int DP>
__global__ __launch_bounds__(256) void k_attn_bf16(AttnArgs a) {
  constexpr int LDK = DP + 8;   // K tile row stride (elements)
  constexpr int LDV = KT + 8;   // V^T tile row stride (elements)
  constexpr int NKC = DP / 32;  // 32-wide chunks of the head dim for QK^T
  constexpr int NET = DP / 16;  // 16-wide output tiles of the head dim (upper bound)
  __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[DP * LDV];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q0 = blockIdx.x * 128 + wave * 32;
  const int N = a.N, d = a.d;
  const int net = (d + 15) / 16;
  const uint16_t* qkv = reinterpret_cast<const uint16_t*>(a.qkv);
  const size_t rb = (size_t)b * N;
  const size_t qoff = (size_t)h * d, koff = (size_t)a.C + h * d, voff = 2 * (size_t)a.C + h * d;
  const u32x4_t z4 = {0u, 0u, 0u, 0u};

  // Q fragments (B operand of S^T): lane holds Q[q][kc*32 + 8*g16 .. +7] for q = q0 + 16g + c16.
  bf16x8_t qf[2][NKC];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int q = q0 + 16 * g + c16;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const int e = kc * 32 + 8 * g16;
      u32x4_t v = (q < N && e < d) ? *reinterpret_cast<const u32x4_t*>(qkv + (rb + q) * a.ldq + qoff + e) : z4;
      qf[g][kc] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  f32x4_t o[2][NET];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int t = 0; t < NET; ++t) o[g][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-INFINITY, -INFINITY}, lrow[2] = {0.f, 0.f};
  const float sl2 = a.scale * 1.4426950408889634f;  // scores in log2 units

  for (int kv0 = 0; kv0 < N; kv0 += KT) {
    __syncthreads();
    for (int c = threadIdx.x; c < KT * (DP / 8); c += 256) {
      const int kr = c / (DP / 8), e = (c % (DP / 8)) * 8, key = kv0 + kr;
      const bool ok = key < N && e < d;
      const u32x4_t kv = ok ? *reinterpret_cast<const u32x4_t*>(qkv + (rb + key) * a.ldq + koff + e) : z4;
      *reinterpret_cast<u32x4_t*>(&Ks[kr * LDK + e]) = kv;
      const u32x4_t vv = ok ? *reinterpret_cast<const u32x4_t*>(qkv + (rb + key) * a.ldq + voff + e) : z4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        Vt[(e + 2 * i) * LDV + kr] = (uint16_t)(vv[i] & 0xffffu);
        Vt[(e + 2 * i + 1) * LDV + kr] = (uint16_t)(vv[i] >> 16);
      }
    }
    __syncthreads();

    // S^T tiles: s[g][t][v] = score(key kv0 + 16t + 4*g16 + v, query q0 + 16g + c16)
    f32x4_t s[2][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      bf16x8_t kf[NKC];
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc)
        kf[kc] = *reinterpret_cast<const bf16x8_t*>(&Ks[(t * 16 + c16) * LDK + kc * 32 + 8 * g16]);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < NKC; ++kc) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kc], qf[g][kc], acc, 0, 0, 0);
        s[g][t] = acc;
      }
    }

    bf16x8_t pb[2][2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int key = kv0 + 16 * t + 4 * g16 + v;
          const float x = key < N ? s[g][t][v] * sl2 : -INFINITY;
          s[g][t][v] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(mrow[g], mx);
      const float alpha = exp2f(mrow[g] - mnew);
      float ls = 0.f;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float p = exp2f(s[g][t][v] - mnew);
          s[g][t][v] = p;
          ls += p;
        }
      ls += __shfl_xor(ls, 16, 64);
      ls += __shfl_xor(ls, 32, 64);
      lrow[g] = lrow[g] * alpha + ls;
      mrow[g] = mnew;
#pragma unroll
      for (int t = 0; t < NET; ++t) o[g][t] *= alpha;
      // B operand of O^T += V^T P^T for key chunk c: keys 32c + 4*g16 + (0..3) and 32c + 16 + 4*g16 + (0..3)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8_t p;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          p[v] = (__bf16)s[g][2 * c][v];
          p[4 + v] = (__bf16)s[g][2 * c + 1][v];
        }
        pb[g][c] = p;
      }
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int t = 0; t < NET; ++t) {
        if (t < net) {
          const uint16_t* vr = &Vt[(t * 16 + c16) * LDV + 32 * c + 4 * g16];
          const u32x2_t lo = *reinterpret_cast<const u32x2_t*>(vr);
          const u32x2_t hi = *reinterpret_cast<const u32x2_t*>(vr + 16);
          const u32x4_t cat = {lo[0], lo[1], hi[0], hi[1]};
          const bf16x8_t va = __builtin_bit_cast(bf16x8_t, cat);
#pragma unroll
          for (int g = 0; g < 2; ++g) o[g][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[g][c], o[g][t], 0, 0, 0);
        }
      }
    }
  }

  // O^T layout: o[g][t][v] = O[query q0 + 16g + c16][e = 16t + 4*g16 + v]
  uint16_t* out = reinterpret_cast<uint16_t*>(a.out);
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int q = q0 + 16 * g + c16;
    if (q >= N) continue;
    const float inv = 1.0f / lrow[g];
#pragma unroll
    for (int t = 0; t < NET; ++t) {
      const int e = 16 * t + 4 * g16;
      if (t < net && e < d) {
        u32x2_t w;
        w[0] = (uint32_t)f2bf(o[g][t][0] * inv) | ((uint32_t)f2bf(o[g][t][1] * inv) << 16);
        w[1] = (uint32_t)f2bf(o[g][t][2] * inv) | ((uint32_t)f2bf(o[g][t][3] * inv) << 16);
        *reinterpret_cast<u32x2_t*>(out + (rb + q) * a.ldo + (size_t)h * d + e) = w;
      }
    }
  }
}

template <int D>
__global__ __launch_bounds__(64) void k_attn_f32(AttnArgs a) {
  constexpr int T32 = 32;
  __shared__ float Ks[T32][D], Vs[T32][D];
  const int lane = threadIdx.x;
  const int b = blockIdx.z, h = blockIdx.y;
  const int q = blockIdx.x * 64 + lane;
  const int N = a.N, d = a.d;
  const float* qkv = reinterpret_cast<const float*>(a.qkv);
  const size_t rb = (size_t)b * N;
  float qv[D], o[D];
#pragma unroll
  for (int e = 0; e < D; ++e) {
    qv[e] = (q < N && e < d) ? qkv[(rb + q) * a.ldq + (size_t)h * d + e] : 0.f;
    o[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int kv0 = 0; kv0 < N; kv0 += T32) {
    __syncthreads();
    for (int i = lane; i < T32 * D; i += 64) {
      const int j = i / D, e = i % D, key = kv0 + j;
      const bool ok = key < N && e < d;
      Ks[j][e] = ok ? qkv[(rb + key) * a.ldq + a.C + (size_t)h * d + e] : 0.f;
      Vs[j][e] = ok ? qkv[(rb + key) * a.ldq + 2 * (size_t)a.C + (size_t)h * d + e] : 0.f;
    }
    __syncthreads();
    float sc[T32];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < T32; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) acc = fmaf(qv[e], Ks[j][e], acc);
      sc[j] = (kv0 + j < N) ? acc * a.scale : -INFINITY;
      mx = fmaxf(mx, sc[j]);
    }
    const float mnew = fmaxf(m, mx);
    const float alpha = expf(m - mnew);
    l *= alpha;
#pragma unroll
    for (int e = 0; e < D; ++e) o[e] *= alpha;
#pragma unroll
    for (int j = 0; j < T32; ++j) {
      const float p = expf(sc[j] - mnew);
      l += p;
#pragma unroll
      for (int e = 0; e < D; ++e) o[e] = fmaf(p, Vs[j][e], o[e]);
    }
    m = mnew;
  }
  if (q < N) {
    float* out = reinterpret_cast<float*>(a.out);
    const float inv = 1.0f / l;
    for (int e = 0; e < d; ++e) out[(rb + q) * a.ldo + (size_t)h * d + e] = o[e] * inv;
  }
}

}  // namespace

hipError_t attention(int dtype, const AttnArgs& a, hipStream_t s) {
  if (a.N <= 0) return hipSuccess;
  if (dtype == DT_BF16) {
    dim3 grid((a.N + 127) / 128, a.H, a.B);
    if (a.d <= 64) FF_LAUNCH(k_attn_bf16<64>, grid, 256, 0, s, a);
    else if (a.d <= 96) FF_LAUNCH(k_attn_bf16<96>, grid, 256, 0, s, a);
    else FF_LAUNCH(k_attn_bf16<128>, grid, 256, 0, s, a);
  } else {
    dim3 grid((a.N + 63) / 64, a.H, a.B);
    if (a.d <= 64) FF_LAUNCH(k_attn_f32<64>, grid, 64, 0, s, a);
    else FF_LAUNCH(k_attn_f32<128>, grid, 64, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ff
