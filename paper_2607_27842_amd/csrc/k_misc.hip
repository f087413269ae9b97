// Normalisation (adaLN-modulated LayerNorm, per-head QK RMSNorm), the modulation /
// time-embedding GEMV, and the once-per-step latent kernels (patchify, sinusoidal
// time embedding, unpatchify fused with the Euler update).
#include "dev_common.h"

namespace ff {

namespace {

// ---- 4-element access helpers (LayerNorm works in 4-element units for both dtypes)
template <int DT> __device__ __forceinline__ void ld4(const void* p, size_t i, float* v);
template <> __device__ __forceinline__ void ld4<DT_F32>(const void* p, size_t i, float* v) {
  float4 w = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p) + i);
  v[0] = w.x; v[1] = w.y; v[2] = w.z; v[3] = w.w;
}
template <> __device__ __forceinline__ void ld4<DT_BF16>(const void* p, size_t i, float* v) {
  uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(p) + i);
  v[0] = __uint_as_float(w.x << 16); v[1] = __uint_as_float(w.x & 0xffff0000u);
  v[2] = __uint_as_float(w.y << 16); v[3] = __uint_as_float(w.y & 0xffff0000u);
}
template <int DT> __device__ __forceinline__ void st4(void* p, size_t i, const float* v);
template <> __device__ __forceinline__ void st4<DT_F32>(void* p, size_t i, const float* v) {
  *reinterpret_cast<float4*>(reinterpret_cast<float*>(p) + i) = make_float4(v[0], v[1], v[2], v[3]);
}
template <> __device__ __forceinline__ void st4<DT_BF16>(void* p, size_t i, const float* v) {
  uint2 w;
  w.x = pack_bf16x2(v[0], v[1]);
  w.y = pack_bf16x2(v[2], v[3]);
  *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(p) + i) = w;
}

// LayerNorm rows: at most 16 4-element units per lane, C <= 64 * 16 * 4 = 4096 (host check)

// Sum over the 64 lanes of a wavefront for the row statistics, every lane receiving it, in
// a fixed order: within each row of 16 lanes by DPP moves (xor 1, xor 2, then the 8- and
// 16-lane mirrors, which pair each partial sum with one covering the other lanes), then the
// four rows by the gfx950 row-pair and half-wavefront swaps (v_permlane16_swap,
// v_permlane32_swap), each adding the even-row (lower-half) value to the odd-row
// (upper-half) one in every lane.  No step goes through the LDS crossbar (the DPP steps
// alone took about 0.2 us off a LayerNorm launch at DiT-XL/2 size against the butterfly of
// six crossbar shuffles).
template <int CTL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row_sum(float v) {
  v += dpp_mov<0xB1>(v);    // quad_perm [1, 0, 3, 2]
  v += dpp_mov<0x4E>(v);    // quad_perm [2, 3, 0, 1]
  v += dpp_mov<0x141>(v);   // row_half_mirror
  v += dpp_mov<0x140>(v);   // row_mirror
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

// One wavefront per row: LN over C (biased variance, no affine), then adaLN modulation.
// The row and its shift / scale vectors are all loaded up front, so the two reductions
// (mean, then variance about it) are the only waits between the loads and the stores.
// 8-element access: one 16-byte load / store for bf16, two for fp32
template <int DT> __device__ __forceinline__ void ld8(const void* p, size_t i, float* v) {
  St<DT>::load(p, i, v);
  if (St<DT>::V == 4) St<DT>::load(p, i + 4, v + 4);
}
template <int DT> __device__ __forceinline__ void st8(void* p, size_t i, const float* v) {
  St<DT>::store(p, i, v);
  if (St<DT>::V == 4) St<DT>::store(p, i + 4, v + 4);
}

template <int DT_IN, int DT_OUT, int U, bool PRE>   // U: 8-element units per lane, C <= 512 U
__global__ __launch_bounds__(256) void k_ln_modulate(LnModArgs a) {
  const int lane = threadIdx.x % 64;
  const int r = blockIdx.x * 4 + threadIdx.x / 64;
  if (r >= a.rows) return;
  const size_t pr = (size_t)a.map.phys(r);
  const int b = a.map.sample(r);
  const int units = a.C / 8;
  const float* sh = a.shift + (size_t)b * a.ldm;
  const float* sc = a.scale + (size_t)b * a.ldm;
  // Every load of the row is issued before any value is used: a lane's units past the row
  // end load unit 0 (in range) and take no part in the arithmetic.  Under the per-unit lane
  // test the loads were serialised: the compiler waited for each unit's values inside the
  // test that the sums below share with it, one memory round trip per unit.
  float v[U][8], s8[U][8], c8[U][8];
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = k * 64 + lane, uc = u < units ? u : 0;
    ld8<DT_IN>(a.in, pr * a.ldi + uc * 8, v[k]);
    ld8<DT_F32>(sh, uc * 8, s8[k]);
    ld8<DT_F32>(sc, uc * 8, c8[k]);
  }
  if (PRE) {
    // the run of drafted layers that precedes this block, from its history sums: the same
    // fmas in the same order as k_draft_sum, one rounding, written back to the stream.
    // The history terms of UB units are all loaded before their fmas (all units up to
    // C = 2048, two at a time above), so they take one round trip per batch rather than
    // one per unit and term.
    constexpr int UB = U <= 4 ? U : 2;
#pragma unroll
    for (int k0 = 0; k0 < U; k0 += UB) {
      float p[UB][kMaxTerms][8];
#pragma unroll
      for (int m = 0; m < kMaxTerms; ++m) {
        if (m < a.pre.n) {
#pragma unroll
          for (int kk = 0; kk < UB; ++kk) {
            const int u = (k0 + kk) * 64 + lane, uc = u < units ? u : 0;
            const size_t i = pr * a.ldi + uc * 8;
            St<DT_F32>::load_nt(a.pre.slot[m], i, p[kk][m]);
            St<DT_F32>::load_nt(a.pre.slot[m], i + 4, p[kk][m] + 4);
          }
        }
      }
#pragma unroll
      for (int kk = 0; kk < UB; ++kk) {
        const int k = k0 + kk, u = k * 64 + lane;
        if (u < units) {
          float f[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) f[j] = 0.0f;
#pragma unroll
          for (int m = 0; m < kMaxTerms; ++m) {
            if (m < a.pre.n) {
#pragma unroll
              for (int j = 0; j < 8; ++j) f[j] = fmaf(a.pre.c[m], p[kk][m][j], f[j]);
            }
          }
#pragma unroll
          for (int j = 0; j < 8; ++j) v[k][j] = St<DT_IN>::rnd(v[k][j] + f[j]);
          st8<DT_IN>(const_cast<void*>(a.in), pr * a.ldi + u * 8, v[k]);
        }
      }
    }
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k)
    if (k * 64 + lane < units) {
#pragma unroll
      for (int j = 0; j < 8; j += 2) s += v[k][j] + v[k][j + 1];
    }
  const float mean = row_sum(s) / (float)a.C;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = k * 64 + lane;
    if (u < units) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float dlt = v[k][j] - mean;
        q += dlt * dlt;
      }
    }
  }
  const float rstd = 1.0f / sqrtf(row_sum(q) / (float)a.C + a.eps);
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = k * 64 + lane;
    if (u < units) {
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (v[k][j] - mean) * rstd * (1.0f + c8[k][j]) + s8[k][j];
      st8<DT_OUT>(a.out, pr * a.ldo + u * 8, o);
    }
  }
}

// One thread per (row, head): in-place RMSNorm over the head's d elements.
template <int DT>
__global__ __launch_bounds__(256) void k_rms_heads(RmsArgs a) {
  using S = St<DT>;
  const long t = (long)blockIdx.x * 256 + threadIdx.x;
  if (t >= (long)a.rows * a.H) return;
  const int r = (int)(t / a.H), h = (int)(t % a.H);
  const size_t base = (size_t)a.map.phys(r) * a.ld + a.col0 + (size_t)h * a.d;
  float ss = 0.f;
  for (int e = 0; e < a.d; e += 4) {
    float v[4];
    ld4<DT>(a.x, base + e, v);
    ss += (v[0] * v[0] + v[1] * v[1]) + (v[2] * v[2] + v[3] * v[3]);
  }
  const float inv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
  for (int e = 0; e < a.d; e += 4) {
    float v[4];
    ld4<DT>(a.x, base + e, v);
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = v[j] * inv * S::ld1(a.g, e + j);
    st4<DT>(a.x, base + e, v);
  }
}

// q and k of a row in one pass: each lane owns one 16-byte chunk of the row's [q | k]
// columns, the LPH = d / V lanes of a head add their sums of squares with xor shuffles
// (fixed order), and every lane rescales its own chunk.  One wavefront covers 64 chunks.
template <int DT, int LPH>
__global__ __launch_bounds__(256) void k_rms_qk(RmsQKArgs a) {
  using S = St<DT>;
  const int lane = threadIdx.x & 63;
  const long wv = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int span = 2 * a.H * a.d;                 // q and k columns
  const int nseg = (span + 64 * S::V - 1) / (64 * S::V);
  const long r = wv / nseg;
  if (r >= a.rows) return;                        // whole wavefront, no barrier below
  const int col = (int)(wv % nseg) * 64 * S::V + lane * S::V;
  const bool on = col < span;
  const size_t base = (size_t)a.map.phys((int)r) * a.ld;
  const int qk = col >= a.H * a.d;
  const int e = (col - qk * a.H * a.d) % a.d;   // a multiple of V: the gain chunk is one access
  const void* g = qk ? a.gk : a.gq;
  float v[S::V], gv[S::V];
  float ss = 0.f;
  if (on) {
    // the gain chunk is requested with the row chunk (read after the reduction, one
    // element at a time, each of its loads waited on its own)
    S::load(a.x, base + col, v);
    S::load(g, e, gv);
#pragma unroll
    for (int j = 0; j < S::V; ++j) ss = fmaf(v[j], v[j], ss);
  }
#pragma unroll
  for (int o = LPH / 2; o >= 1; o /= 2) ss += __shfl_xor(ss, o, 64);
  if (!on) return;
  const float inv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
#pragma unroll
  for (int j = 0; j < S::V; ++j) v[j] = v[j] * inv * gv[j];
  const Rope& ro = a.rope;
  if (ro.axes[0] + ro.axes[1] + ro.axes[2]) {
    // the row's token n within its sample; image rows carry (frame, row, column) ids
    const int n = a.map.off + (int)(r % a.map.n_seg);
    if (n >= ro.n_txt) {
      const int t = n - ro.n_txt;
      const float pos[3] = {(float)(t / (ro.Hp * ro.Wp)), (float)((t / ro.Wp) % ro.Hp), (float)(t % ro.Wp)};
#pragma unroll
      for (int j = 0; j < S::V; j += 2) {   // e + j is even: a lane holds whole pairs
        int p = e + j, ax = 0;
        if (p >= ro.axes[0]) { p -= ro.axes[0]; ax = 1; if (p >= ro.axes[1]) { p -= ro.axes[1]; ax = 2; } }
        // selects, not ro.axes[ax] / pos[ax]: a lane-varying index into the argument block
        // became a memory load (and a wait) per pair
        const int da = ax == 0 ? ro.axes[0] : (ax == 1 ? ro.axes[1] : ro.axes[2]);
        const float ps = ax == 0 ? pos[0] : (ax == 1 ? pos[1] : pos[2]);
        const float w = exp2f(-(float)p / (float)da * ro.log2_theta);   // theta^(-2i/da), p = 2i
        float sn, cs;
        sincosf(ps * w, &sn, &cs);
        const float x0 = v[j], x1 = v[j + 1];
        v[j] = x0 * cs - x1 * sn;
        v[j + 1] = x0 * sn + x1 * cs;
      }
    }
  }
  S::store(a.x, base + col, v);
}

constexpr int kGemvTileB = 8;   // samples per launch of the generic tile
constexpr int kGemvRows = 4;     // output features per wavefront
constexpr int kGemvKC = 1024;    // K chunk of the activations staged in LDS

// y[b, n] for 16 consecutive n per workgroup (4 per wavefront).  The activations x[b, k]
// (after the optional SiLU) are staged in LDS once per K chunk and shared by all rows.
// Per chunk, every lane first issues all of its 16-byte weight loads (consecutive lanes
// -> consecutive chunks of a row) and every thread all of its activation loads, so the
// chunk costs one memory round trip; then one sum per (row, sample) is accumulated.
template <int DT>
__device__ __forceinline__ void gemv_tile(const GemvArgs a, int blk) {
  using S = St<DT>;
  constexpr int kPer = kGemvKC / S::V / 64;   // weight chunks per lane per K chunk
  extern __shared__ float xs[];               // [B][kGemvKC]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = (blk * 4 + wave) * kGemvRows;
  float acc[kGemvRows][kGemvTileB];
#pragma unroll
  for (int r = 0; r < kGemvRows; ++r)
#pragma unroll
    for (int b = 0; b < kGemvTileB; ++b) acc[r][b] = 0.f;
  for (int k0 = 0; k0 < a.K; k0 += kGemvKC) {
    const int kc = min(kGemvKC, a.K - k0);
    // weight loads first (they do not depend on the activations) ...
    float w[kPer][kGemvRows][S::V];
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int c = lane + 64 * p;
#pragma unroll
      for (int r = 0; r < kGemvRows; ++r) {
        if (c * S::V < kc && n0 + r < a.Nout) {
          S::load(a.W, (size_t)(n0 + r) * a.K + k0 + c * S::V, w[p][r]);
        } else {
#pragma unroll
          for (int j = 0; j < S::V; ++j) w[p][r][j] = 0.f;
        }
      }
    }
    // ... then every sample's activation chunk (one float4 per thread and sample, all
    // loads issued before any is stored) into LDS
    float4 xv4[kGemvTileB];
    const int k4 = threadIdx.x * 4;   // 256 threads x 4 = kGemvKC
#pragma unroll
    for (int b = 0; b < kGemvTileB; ++b)
      if (b < a.B && k4 < kc) xv4[b] = *reinterpret_cast<const float4*>(a.x + (size_t)b * a.ldx + k0 + k4);
    __syncthreads();   // the previous chunk's LDS reads are done
#pragma unroll
    for (int b = 0; b < kGemvTileB; ++b) {
      if (b < a.B && k4 < kc) {
        float4 v = xv4[b];
        if (a.silu_in) { v.x = silu_f(v.x); v.y = silu_f(v.y); v.z = silu_f(v.z); v.w = silu_f(v.w); }
        *reinterpret_cast<float4*>(&xs[b * kGemvKC + k4]) = v;
      }
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int c = lane + 64 * p;
      if (c * S::V >= kc) break;
#pragma unroll
      for (int b = 0; b < kGemvTileB; ++b) {
        if (b < a.B) {
          float xv[S::V];
#pragma unroll
          for (int j = 0; j < S::V; j += 4) {
            const float4 q = *reinterpret_cast<const float4*>(&xs[b * kGemvKC + c * S::V + j]);
            xv[j] = q.x; xv[j + 1] = q.y; xv[j + 2] = q.z; xv[j + 3] = q.w;
          }
#pragma unroll
          for (int r = 0; r < kGemvRows; ++r)
#pragma unroll
            for (int j = 0; j < S::V; ++j) acc[r][b] = fmaf(xv[j], w[p][r][j], acc[r][b]);
        }
      }
    }
  }
  // Cross-lane sums of the kGemvRows * B partials: one transposed pass through LDS (each
  // lane writes its partials, lane v then adds column v over the 64 lanes in order) instead
  // of one 6-step butterfly per value.
  __shared__ float red[4][kGemvRows * kGemvTileB][65];
#pragma unroll
  for (int r = 0; r < kGemvRows; ++r)
#pragma unroll
    for (int b = 0; b < kGemvTileB; ++b) red[wave][r * kGemvTileB + b][lane] = acc[r][b];
  __syncthreads();
  if (lane < kGemvRows * kGemvTileB) {
    const int r = lane / kGemvTileB, b = lane % kGemvTileB, n = n0 + r;
    if (b < a.B && n < a.Nout) {
      float sum = 0.f;
      for (int l = 0; l < 64; ++l) sum += red[wave][lane][l];
      float y = sum + S::ld1(a.bias, n);
      if (a.silu_out) y = silu_f(y);
      if (a.add) y += a.add[(size_t)b * a.ldadd + n];
      a.y[(size_t)b * a.ldy + n] = y;
    }
  }
}

// bf16 weights, B <= 32: y[b, n0..n0+15] on v_mfma_f32_16x16x32_bf16.  The fp32
// activations enter as bf16 hi + lo parts (x = hi + lo to ~2^-17 relative), split by each
// lane as it loads them, or read from a split made beforehand (xs; the large modulation
// batches, whose thousands of workgroups would otherwise each split the same x): MFMA
// rows 0-7 carry hi of samples 0-7 and rows 8-15 lo, so one instruction covers both halves and output rows b and b+8 are added at the
// end.  The four wavefronts take interleaved 32-wide K steps and their 16x16 partial
// tiles are summed through LDS in wavefront order.  16x16x32 layouts: A lane l holds row
// l%16, k = 8*(l/16)+0..7; B lane l holds column l%16, same k; D lane l holds column
// l%16, rows 4*(l/16)+0..3.
constexpr int kMvU = 4;   // K steps per wavefront whose loads are issued together

// The 8 activations x[k..k+7] (SiLU first if silu_in) as bf16 hi parts, or as the bf16
// rounding of what hi leaves (lo).
__device__ __forceinline__ u32x4_t split8(const float* x, int silu_in, bool lo_part) {
  const f32x4_t v0 = *reinterpret_cast<const f32x4_t*>(x);
  const f32x4_t v1 = *reinterpret_cast<const f32x4_t*>(x + 4);
  u32x4_t r;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float a0 = j < 2 ? v0[2 * j] : v1[2 * j - 4], a1 = j < 2 ? v0[2 * j + 1] : v1[2 * j - 3];
    if (silu_in) { a0 = silu_f(a0); a1 = silu_f(a1); }
    uint16_t h0 = f2bf(a0), h1 = f2bf(a1);
    if (lo_part) { h0 = f2bf(a0 - bf2f(h0)); h1 = f2bf(a1 - bf2f(h1)); }
    r[j] = (uint32_t)h0 | ((uint32_t)h1 << 16);
  }
  return r;
}

// NG groups of 8 samples share each weight load: group g holds samples 8g..8g+7 (its
// split in xs rows 16g..16g+15) and its own accumulator tile.
template <int NG>
__device__ __forceinline__ void gemv_mfma_tile(const GemvArgs a, int blk) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blk * 16;
  const int rc = lane & 15, kq = (lane >> 4) * 8;
  const int n = n0 + rc;
  const bool nok = n < a.Nout;
  const uint16_t* wrow = reinterpret_cast<const uint16_t*>(a.W) + (size_t)(nok ? n : 0) * a.K;
  const bool lo_part = rc >= 8;
  const int nks = (a.K + 31) / 32;
  const u32x4_t z4 = {0u, 0u, 0u, 0u};
  f32x4_t acc[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) acc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int ks0 = wave; ks0 < nks; ks0 += 4 * kMvU) {
    u32x4_t wv[kMvU], xv[NG][kMvU];
#pragma unroll
    for (int u = 0; u < kMvU; ++u) {
      const int k = (ks0 + 4 * u) * 32 + kq;
      const bool kin = ks0 + 4 * u < nks && k < a.K;   // K % 8 == 0: a lane's 8 are all in or out
      wv[u] = (kin && nok) ? *reinterpret_cast<const u32x4_t*>(wrow + k) : z4;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int b = 8 * g + (rc & 7);   // sample of this lane's A row (ldx 0: one shared row)
        if (!(kin && b < a.B)) xv[g][u] = z4;
        else if (a.xs) xv[g][u] = *reinterpret_cast<const u32x4_t*>(a.xs + (size_t)(16 * g + rc) * a.K + k);
        else xv[g][u] = split8(a.x + (size_t)b * a.ldx + k, a.silu_in, lo_part);
      }
    }
#pragma unroll
    for (int u = 0; u < kMvU; ++u)
#pragma unroll
      for (int g = 0; g < NG; ++g)
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, xv[g][u]),
                                                         __builtin_bit_cast(bf16x8_t, wv[u]), acc[g], 0, 0, 0);
  }
  __shared__ float red[4][64][4 * NG];
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wave][lane][4 * g + j] = acc[g][j];
  __syncthreads();
  if (threadIdx.x < 128) {
    const int ob = threadIdx.x >> 4, on = threadIdx.x & 15;   // output (sample in group, column)
    const int lh = (ob >> 2) * 16 + on, ll = ((ob >> 2) + 2) * 16 + on, j = ob & 3;
    const int nn = n0 + on;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      float hi = 0.f, lw = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) { hi += red[w][lh][4 * g + j]; lw += red[w][ll][4 * g + j]; }
      const int b = 8 * g + ob;
      if (b < a.B && nn < a.Nout) {
        float y = (hi + lw) + St<DT_BF16>::ld1(a.bias, nn);
        if (a.silu_out) y = silu_f(y);
        if (a.add) y += a.add[(size_t)b * a.ldadd + nn];
        a.y[(size_t)b * a.ldy + nn] = y;
      }
    }
  }
}

template <int NG>
__global__ __launch_bounds__(256) void k_gemv_mfma(GemvArgs a) { gemv_mfma_tile<NG>(a, blockIdx.x); }

template <int NG>
__global__ __launch_bounds__(256) void k_gemv_mfma_batch(GemvBatch bt) {
  const GemvJob j = bt.job[blockIdx.y];
  if ((int)blockIdx.x * 16 >= j.Nout) return;   // whole workgroup: no barrier skipped
  const GemvArgs a{bt.x, bt.ldx, bt.silu_in, j.W, j.bias, j.Nout, bt.K, bt.B, j.y, j.ldy, 0, nullptr, 0, bt.xs};
  gemv_mfma_tile<NG>(a, blockIdx.x);
}

template <int DT>
__global__ __launch_bounds__(256) void k_gemv(GemvArgs a) { gemv_tile<DT>(a, blockIdx.x); }

// Several independent GEMVs over the same activations in one launch (blockIdx.y = job):
// the modulation vectors of every exact layer of a step, so that the weight streams of
// all of them share one grid instead of one small launch each.
template <int DT>
__global__ __launch_bounds__(256) void k_gemv_batch(GemvBatch bt) {
  const GemvJob j = bt.job[blockIdx.y];
  if ((int)blockIdx.x * 4 * kGemvRows >= j.Nout) return;   // whole workgroup: no barrier skipped
  const GemvArgs a{bt.x, bt.ldx, bt.silu_in, j.W, j.bias, j.Nout, bt.K, bt.B, j.y, j.ldy, 0, nullptr, 0};
  gemv_tile<DT>(a, blockIdx.x);
}

__global__ void k_time_embed(double s, float* phi) {
  const int k = threadIdx.x;  // 0..127
  const double f = exp(-log(10000.0) * (double)k / 128.0);
  phi[k] = (float)cos(s * f);
  phi[128 + k] = (float)sin(s * f);
}

__global__ void k_time_embed_steps(double T, int n, float* phi) {
  const int k = threadIdx.x, i = blockIdx.x;   // 0..127, step
  if (i >= n) return;
  const double s = 1000.0 * (1.0 - (double)i / T);
  const double f = exp(-log(10000.0) * (double)k / 128.0);
  phi[(size_t)i * 256 + k] = (float)cos(s * f);
  phi[(size_t)i * 256 + 128 + k] = (float)sin(s * f);
}

__global__ void k_cond_split(const float* u, const float* cond, int nsteps, int B, int C, uint16_t* xs, float* cs,
                             uint16_t* zb, int nzb) {
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (zb && idx < nzb) zb[idx] = 0;
  const int G8 = xs ? (B + 7) / 8 * 8 : B;   // rows per step, absent samples included
  if (idx >= (long)nsteps * G8 * C) return;
  const int k = (int)(idx % C);
  const long ib = idx / C;
  const int b = (int)(ib % G8), i = (int)(ib / G8);
  // c_t = cond + u and its SiLU as the per-step path forms them (fp32)
  const float v = b < B ? silu_f(cond[(size_t)b * C + k] + u[(size_t)i * C + k]) : 0.f;
  if (xs) {
    uint16_t* x = xs + (size_t)i * 2 * G8 * C;   // 16 rows per group of 8
    const int r = 16 * (b / 8) + b % 8;
    const uint16_t h = f2bf(v);
    x[(size_t)r * C + k] = h;
    x[(size_t)(r + 8) * C + k] = f2bf(v - bf2f(h));
  } else {
    cs[((size_t)i * B + b) * C + k] = v;
  }
}

template <int DT>
__global__ void k_mod_combine(const float* __restrict__ out, int N, const void* __restrict__ bias,
                              float* __restrict__ dst, int ldy, int nb, int B) {
  const int n4 = N / 4;
  const long idx = (long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long)nb * B * n4) return;
  const int n = (int)(idx % n4) * 4;
  const long jb = idx / n4;
  const int b = (int)(jb % B), j = (int)(jb / B);
  const int R16 = 16 * ((B + 7) / 8), r = j * R16 + 16 * (b / 8) + b % 8;
  const f32x4_t hi = *reinterpret_cast<const f32x4_t*>(out + (size_t)r * N + n);
  const f32x4_t lo = *reinterpret_cast<const f32x4_t*>(out + (size_t)(r + 8) * N + n);
  float bv[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) bv[e] = St<DT>::ld1(bias, n + e);
  f32x4_t y;
#pragma unroll
  for (int e = 0; e < 4; ++e) y[e] = (hi[e] + lo[e]) + bv[e];
  *reinterpret_cast<f32x4_t*>(dst + (size_t)jb * ldy + n) = y;
}

__global__ void k_silu_rows(const float* x, float* y, int B, int n, uint16_t* xs) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)B * n) return;
  const float v = silu_f(x[i]);
  y[i] = v;
  if (xs) {   // the bf16 hi / lo split the MFMA GEMVs read (as split8 makes it)
    const int b = (int)(i / n), k = (int)(i % n);
    const int r = 16 * (b / 8) + b % 8;   // group b/8: hi rows 16g..16g+7, lo 16g+8..
    const uint16_t h = f2bf(v);
    xs[(size_t)r * n + k] = h;
    xs[(size_t)(r + 8) * n + k] = f2bf(v - bf2f(h));
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_patchify(const float* __restrict__ x, void* __restrict__ out, PatchGeom g) {
  const int Fp = g.F / g.pt, Hp = g.H / g.ph, Wp = g.W / g.pw;
  const int P = g.pt * g.ph * g.pw * g.lat_c;
  const long n_img = (long)Fp * Hp * Wp;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)g.B * n_img * P) return;
  const int feat = (int)(i % P);
  const long row = i / P;
  const int b = (int)(row / n_img);
  const int tok = (int)(row % n_img);
  const int wx = tok % Wp, hy = (tok / Wp) % Hp, f = tok / (Wp * Hp);
  const int bl = g.lat_B ? b % g.lat_B : b;   // the latent this row reads (guided pairs share one)
  // feature order (channel, dt, dy, dx)
  const int c = feat % g.pw, bb = (feat / g.pw) % g.ph, a = (feat / (g.pw * g.ph)) % g.pt;
  const int ch = feat / (g.pw * g.ph * g.pt);
  const size_t src = ((((size_t)bl * g.lat_c + ch) * g.F + (f * g.pt + a)) * g.H + (hy * g.ph + bb)) * g.W +
                     (wx * g.pw + c);
  St<DT>::st1(out, (size_t)i, x[src]);
}

__global__ __launch_bounds__(256) void k_unpatchify_euler(const float* __restrict__ yv, float* __restrict__ x,
                                                          float dt, PatchGeom g) {
  const long n = (long)(g.lat_B ? g.lat_B : g.B) * g.lat_c * g.F * g.H * g.W;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const int xx = (int)(i % g.W);
  const int yy = (int)((i / g.W) % g.H);
  const int ff = (int)((i / ((long)g.W * g.H)) % g.F);
  const int ch = (int)((i / ((long)g.W * g.H * g.F)) % g.lat_c);
  const int b = (int)(i / ((long)g.W * g.H * g.F * g.lat_c));
  const int Fp = g.F / g.pt, Hp = g.H / g.ph, Wp = g.W / g.pw;
  const int P = g.pt * g.ph * g.pw * g.lat_c;
  const long tok = ((long)(ff / g.pt) * Hp + yy / g.ph) * Wp + xx / g.pw;
  // feature order (dt, dy, dx, channel)
  const int feat = (((ff % g.pt) * g.ph + yy % g.ph) * g.pw + xx % g.pw) * g.lat_c + ch;
  const long n_img = (long)Fp * Hp * Wp;
  float v = yv[((long)b * n_img + tok) * P + feat];
  if (g.cfg_half) {   // guidance: v_u + s (v_c - v_u), v_c from row b, v_u from row b + half
    const float vu = yv[((long)(b + g.cfg_half) * n_img + tok) * P + feat];
    v = vu + g.cfg_scale * (v - vu);
  }
  x[i] = x[i] + dt * v;
}


// Sum of NP per-lane values over the 64 lanes of a wavefront, by recursive halving: at the
// step with stride s, a lane keeps one half of its values (the upper half if lane & s),
// adds the partner's copy of that half, and hands over the other half.  After log2(NP)
// steps every lane holds one output, o = lane / (64 / NP); the remaining strides sum the
// lanes that share it.  63 shuffles for NP = 64 instead of 6 NP.
template <int NP>
__device__ __forceinline__ float wave_reduce_outputs(float (&v)[NP], int lane) {
  static_assert(NP >= 1 && NP <= 64 && (NP & (NP - 1)) == 0, "power of two");
#pragma unroll
  for (int n = NP, s = 32; n > 1; n /= 2, s /= 2) {
    const bool upper = (lane & s) != 0;
#pragma unroll
    for (int k = 0; k < n / 2; ++k) {
      const float send = upper ? v[k] : v[k + n / 2];
      const float recv = __shfl_xor(send, s, 64);
      v[k] = (upper ? v[k + n / 2] : v[k]) + recv;
    }
  }
  float r = v[0];
#pragma unroll
  for (int s = 32 / NP; s > 0; s /= 2) r += __shfl_xor(r, s, 64);
  return r;
}

// Final weights up to this size are read straight from the caches by every wavefront;
// larger ones (FLUX-like: 384 KB) make that L2-bound, and the GEMM path, which reuses the
// weight across a tile, is faster there.
constexpr size_t kFinalMaxWeightBytes = 64 * 1024;

template <int DT, int U, int NP>   // U: 4-element units per lane, NP: outputs per token
__global__ __launch_bounds__(256) void k_final_layer(FinalArgs a) {
  using S = St<DT>;
  const int lane = threadIdx.x % 64;
  const int r = blockIdx.x * 4 + threadIdx.x / 64;
  if (r >= a.rows) return;   // r is per wavefront: the whole wave leaves together
  const size_t pr = (size_t)a.map.phys(r);
  const int b = a.map.sample(r);
  const int units = a.C / 4;
  const float* sh = a.shift + (size_t)b * a.ldm;
  const float* sc = a.scale + (size_t)b * a.ldm;
  float v[U][4];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = k * 64 + lane;
    if (u < units) ld4<DT>(a.in, pr * a.ldi + u * 4, v[k]);
  }
#pragma unroll
  for (int k = 0; k < U; ++k)
    if (k * 64 + lane < units) s += (v[k][0] + v[k][1]) + (v[k][2] + v[k][3]);
  const float mean = row_sum(s) / (float)a.C;
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < U; ++k)
    if (k * 64 + lane < units) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float dlt = v[k][j] - mean;
        q += dlt * dlt;
      }
    }
  const float rstd = 1.0f / sqrtf(row_sum(q) / (float)a.C + a.eps);
  // the modulated row, rounded to the model dtype as ln_modulate stores it
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const int u = k * 64 + lane;
    if (u < units) {
      const float4 s4 = *reinterpret_cast<const float4*>(sh + u * 4);
      const float4 c4 = *reinterpret_cast<const float4*>(sc + u * 4);
      v[k][0] = St<DT>::rnd((v[k][0] - mean) * rstd * (1.0f + c4.x) + s4.x);
      v[k][1] = St<DT>::rnd((v[k][1] - mean) * rstd * (1.0f + c4.y) + s4.y);
      v[k][2] = St<DT>::rnd((v[k][2] - mean) * rstd * (1.0f + c4.z) + s4.z);
      v[k][3] = St<DT>::rnd((v[k][3] - mean) * rstd * (1.0f + c4.w) + s4.w);
    }
  }
  // outputs in groups of at most 32 (register budget), each reduced over the wavefront
  constexpr int NG = NP > 32 ? 32 : NP;
  constexpr int LPO = 64 / NG;   // lanes per output after the reduction
  const PatchGeom& g = a.g;
  const int Hp = g.H / g.ph, Wp = g.W / g.pw;
  const int n_img = (g.F / g.pt) * Hp * Wp;
  const int tok = r - b * n_img;
  const int wx = tok % Wp, hy = (tok / Wp) % Hp, f = tok / (Wp * Hp);
#pragma unroll
  for (int og = 0; og < NP; og += NG) {
    float acc[NG];
#pragma unroll
    for (int o = 0; o < NG; ++o) acc[o] = 0.f;
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int u = k * 64 + lane;
      if (u < units) {
#pragma unroll
        for (int o = 0; o < NG; ++o) {
          float w[4];
          ld4<DT>(a.W, (size_t)(og + o) * a.C + u * 4, w);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[o] = fmaf(v[k][j], w[j], acc[o]);
        }
      }
    }
    const float sum = wave_reduce_outputs<NG>(acc, lane);
    if (lane % LPO == 0) {
      const int o = og + lane / LPO;
      const float val = sum + S::ld1(a.bias, o);
      // unpatchify: output o of token (b, tok) is latent pixel (ch, f pt + da, hy ph + dy, wx pw + dx)
      const int ch = o % g.lat_c, dx = (o / g.lat_c) % g.pw, dy = (o / (g.lat_c * g.pw)) % g.ph;
      const int da = o / (g.lat_c * g.pw * g.ph);
      const size_t idx = ((((size_t)b * g.lat_c + ch) * g.F + (f * g.pt + da)) * g.H + (hy * g.ph + dy)) * g.W +
                         (wx * g.pw + dx);
      a.x[idx] = a.x[idx] + a.dt * val;
    }
  }
}

// The same final layer in bf16 on v_mfma_f32_32x32x16_bf16, for at most 32 outputs per
// token and C <= kFinMfmaMaxC (C % 16 == 0).  A workgroup of 8 wavefronts takes ROWS token
// rows: each wavefront loads its ROWS / 8 rows at once, normalises them (LN + modulation,
// rounded to bf16 as ln_modulate stores it) into an LDS tile [ROWS][C + 8]; wavefront w
// then accumulates the 16-wide k steps w, w + 8, ... of v^T = W a^T, with its W fragments
// loaded at the start (rows of W past P read as zero; the MFMA's 32 token columns repeat
// the ROWS rows); the eight partial sums meet in LDS in wavefront order, and wavefront 0
// adds the bias and applies the Euler update to the latent values it read at the start.
// W is read once per ROWS tokens instead of once per token.
constexpr int kFinMfmaMaxC = 1536;

// latent index of output o (feature order (dt, dy, dx, ch)) of image token tok of sample b
__device__ __forceinline__ size_t fin_pixel(const PatchGeom& g, int b, int tok, int o) {
  const int Hp = g.H / g.ph, Wp = g.W / g.pw;
  const int wx = tok % Wp, hy = (tok / Wp) % Hp, f = tok / (Wp * Hp);
  const int ch = o % g.lat_c, dx = (o / g.lat_c) % g.pw, dy = (o / (g.lat_c * g.pw)) % g.ph;
  const int da = o / (g.lat_c * g.pw * g.ph);
  return ((((size_t)b * g.lat_c + ch) * g.F + (f * g.pt + da)) * g.H + (hy * g.ph + dy)) * g.W + (wx * g.pw + dx);
}

template <int ROWS>   // token rows per workgroup: 8 or 16
__global__ __launch_bounds__(512) void k_final_mfma(FinalArgs a) {
  constexpr int kFinMfmaRows = ROWS;
  static_assert(ROWS == 8 || ROWS == 16, "rows per workgroup");
  constexpr int LDA = kFinMfmaMaxC + 8;         // LDS row pitch (elements): 16-byte aligned rows
  constexpr int U8 = kFinMfmaMaxC / 8 / 64;     // 8-element units per lane and row
  constexpr int KW = kFinMfmaMaxC / 16 / 8;     // k steps per wavefront
  constexpr int RPW = kFinMfmaRows / 8;         // rows per wavefront
  constexpr int kXch = 7 * 16 * 64 * 2;         // the exchange of wavefronts 1-7 (uint16 units)
  __shared__ __attribute__((aligned(16))) uint16_t sA[kFinMfmaRows * LDA > kXch ? kFinMfmaRows * LDA : kXch];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r0 = blockIdx.x * kFinMfmaRows;
  const int C = a.C, units = C / 8, nks = C / 16;
  const int P = a.g.pt * a.g.ph * a.g.pw * a.g.lat_c;
  const uint16_t* Wt = reinterpret_cast<const uint16_t*>(a.W);
  const uint16_t* in = reinterpret_cast<const uint16_t*>(a.in);
  const u32x4_t z4 = {0u, 0u, 0u, 0u};
  // wavefront 0 reads the latent values it will update, and their output biases, first:
  // lane l, output 8 (v/4) + 4 (l/32) + v%4 of token row l%32 (a bias read at the end
  // made each of the 16 updates wait for its own load)
  const int n_img = (a.g.F / a.g.pt) * (a.g.H / a.g.ph) * (a.g.W / a.g.pw);
  const int me = lane & 31, re = r0 + me;
  const bool eout = wave == 0 && me < kFinMfmaRows && re < a.rows;
  float xv[16];
  uint16_t bv[16];   // raw bf16: converted where it is used, so no load waits here
  size_t xi[16];
  if (eout) {
    const int b = a.map.sample(re), tok = re - b * n_img;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int o = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
      xi[v] = o < P ? fin_pixel(a.g, b, tok, o) : 0;
      xv[v] = o < P ? a.x[xi[v]] : 0.f;
      bv[v] = o < P ? reinterpret_cast<const uint16_t*>(a.bias)[o] : (uint16_t)0;
    }
  }
  // this wavefront's rows, all loads in flight together
  u32x4_t raw[RPW][U8];
#pragma unroll
  for (int j = 0; j < RPW; ++j) {
    const int r = r0 + wave * RPW + j;
    const size_t pr = r < a.rows ? (size_t)a.map.phys(r) : 0;
#pragma unroll
    for (int k = 0; k < U8; ++k) {
      const int u = k * 64 + lane;
      raw[j][k] = (r < a.rows && u < units) ? *reinterpret_cast<const u32x4_t*>(in + pr * a.ldi + u * 8) : z4;
    }
  }
  // W fragments of this wavefront's k steps: lane l holds output l%32, k 16 s + 8 (l/32) + 0..7
  bf16x8_t wf[KW];
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    const int s = wave + 8 * j, n = lane & 31;
    const u32x4_t v = (s < nks && n < P) ? *reinterpret_cast<const u32x4_t*>(Wt + (size_t)n * C + 16 * s + 8 * (lane >> 5)) : z4;
    wf[j] = __builtin_bit_cast(bf16x8_t, v);
  }
  // LN + modulation (rows past the end are left unwritten: their outputs are never stored)
  int bcur = -1;
  float s8[U8][8], c8[U8][8];
#pragma unroll
  for (int j = 0; j < RPW; ++j) {
    const int rr = wave * RPW + j, r = r0 + rr;
    if (r >= a.rows) break;
    const int b = a.map.sample(r);
    if (b != bcur) {   // the shift / scale of this row's sample (uniform per wavefront)
      bcur = b;
      const float* sh = a.shift + (size_t)b * a.ldm;
      const float* sc = a.scale + (size_t)b * a.ldm;
#pragma unroll
      for (int k = 0; k < U8; ++k) {
        const int u = k * 64 + lane;
        if (u < units) {
          St<DT_F32>::load(sh, u * 8, s8[k]);
          St<DT_F32>::load(sh, u * 8 + 4, s8[k] + 4);
          St<DT_F32>::load(sc, u * 8, c8[k]);
          St<DT_F32>::load(sc, u * 8 + 4, c8[k] + 4);
        }
      }
    }
    float v[U8][8];
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < U8; ++k) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[k][2 * q] = __uint_as_float(raw[j][k][q] << 16);
        v[k][2 * q + 1] = __uint_as_float(raw[j][k][q] & 0xffff0000u);
      }
      if (k * 64 + lane < units) {
#pragma unroll
        for (int q = 0; q < 8; q += 2) s += v[k][q] + v[k][q + 1];
      }
    }
    const float mean = row_sum(s) / (float)C;
    float qv = 0.f;
#pragma unroll
    for (int k = 0; k < U8; ++k)
      if (k * 64 + lane < units) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float dlt = v[k][q] - mean;
          qv += dlt * dlt;
        }
      }
    const float rstd = 1.0f / sqrtf(row_sum(qv) / (float)C + a.eps);
#pragma unroll
    for (int k = 0; k < U8; ++k) {
      const int u = k * 64 + lane;
      if (u < units) {
        float o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = (v[k][q] - mean) * rstd * (1.0f + c8[k][q]) + s8[k][q];
        St<DT_BF16>::store(sA + rr * LDA, u * 8, o);
      }
    }
  }
  __syncthreads();
  // lane l: token row (l%32) % ROWS; D[v] holds output 8 (v/4) + 4 (l/32) + v%4
  f32x16_t acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.f;
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    const int s = wave + 8 * j;
    if (s < nks) {
      const bf16x8_t af = *reinterpret_cast<const bf16x8_t*>(sA + (lane & (kFinMfmaRows - 1)) * LDA + 16 * s + 8 * (lane >> 5));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[j], af, acc, 0, 0, 0);
    }
  }
  __syncthreads();   // every wavefront's tile reads are done: the tile becomes the exchange
  float* red = reinterpret_cast<float*>(sA);
  static_assert(7 * 16 * 64 * 4 <= sizeof(sA), "exchange space");
  if (wave > 0) {
#pragma unroll
    for (int v = 0; v < 16; ++v) red[((wave - 1) * 16 + v) * 64 + lane] = acc[v];
  }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 1; w < 8; ++w)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] += red[((w - 1) * 16 + v) * 64 + lane];
  if (!eout) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int o = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    if (o < P) a.x[xi[v]] = xv[v] + a.dt * (acc[v] + bf2f(bv[v]));
  }
}

}  // namespace

hipError_t ln_modulate(int dtype, const LnModArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int grid = cdiv(a.rows, 4);
  const int units = cdiv(a.C / 8, 64);   // 8-element units per lane (C % 8 == 0, C <= 4096 checked on the host)
  if (a.pre.n < 0 || a.pre.n > kMaxTerms || (a.pre.n > 0 && a.in_f32)) return hipErrorInvalidValue;
#define FF_LN(U)                                                                                 \
  do {                                                                                           \
    if (dtype == DT_BF16) {                                                                      \
      if (a.in_f32) FF_LAUNCH((k_ln_modulate<DT_F32, DT_BF16, U, false>), grid, 256, 0, s, a);   \
      else if (a.pre.n) FF_LAUNCH((k_ln_modulate<DT_BF16, DT_BF16, U, true>), grid, 256, 0, s, a); \
      else FF_LAUNCH((k_ln_modulate<DT_BF16, DT_BF16, U, false>), grid, 256, 0, s, a);           \
    } else if (a.pre.n) {                                                                        \
      FF_LAUNCH((k_ln_modulate<DT_F32, DT_F32, U, true>), grid, 256, 0, s, a);                   \
    } else {                                                                                     \
      FF_LAUNCH((k_ln_modulate<DT_F32, DT_F32, U, false>), grid, 256, 0, s, a);                  \
    }                                                                                            \
  } while (0)
  if (units <= 1) FF_LN(1);
  else if (units <= 3) FF_LN(3);
  else if (units <= 4) FF_LN(4);
  else if (units <= 6) FF_LN(6);
  else FF_LN(8);
#undef FF_LN
  return hipGetLastError();
}

hipError_t rms_heads(int dtype, const RmsArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int grid = cdiv((long)a.rows * a.H, 256);
  if (dtype == DT_BF16) FF_LAUNCH(k_rms_heads<DT_BF16>, grid, 256, 0, s, a);
  else FF_LAUNCH(k_rms_heads<DT_F32>, grid, 256, 0, s, a);
  return hipGetLastError();
}

hipError_t rms_qk(int dtype, const RmsQKArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int V = dtype == DT_BF16 ? 8 : 4;
  const int lph = a.d / V;
  const bool fast = a.d % V == 0 && (lph == 8 || lph == 16 || lph == 32) && (64 * V) % a.d == 0;
  if (!fast) {   // per-head thread kernel, q then k
    RmsArgs q{a.x, a.ld, a.map, a.rows, a.H, a.d, 0, a.gq, a.eps};
    hipError_t e = rms_heads(dtype, q, s);
    if (e != hipSuccess) return e;
    RmsArgs k{a.x, a.ld, a.map, a.rows, a.H, a.d, a.H * a.d, a.gk, a.eps};
    return rms_heads(dtype, k, s);
  }
  const int nseg = cdiv(2 * a.H * a.d, 64 * V);
  const int grid = cdiv((long)a.rows * nseg, 4);
#define FF_RMS(LPH)                                                            \
  do {                                                                         \
    if (dtype == DT_BF16) FF_LAUNCH((k_rms_qk<DT_BF16, LPH>), grid, 256, 0, s, a); \
    else FF_LAUNCH((k_rms_qk<DT_F32, LPH>), grid, 256, 0, s, a);              \
  } while (0)
  if (lph == 8) FF_RMS(8);
  else if (lph == 16) FF_RMS(16);
  else FF_RMS(32);
#undef FF_RMS
  return hipGetLastError();
}

hipError_t gemv(int dtype, const GemvArgs& a, hipStream_t s) {
  if (a.B < 1 || a.B > kGemvMaxB) return hipErrorInvalidValue;
  if (dtype == DT_BF16) {
    if (a.K % 8) return hipErrorInvalidValue;
    const int grid = cdiv(a.Nout, 16), ng = cdiv(a.B, 8);
    if (ng == 1) FF_LAUNCH(k_gemv_mfma<1>, grid, 256, 0, s, a);
    else if (ng == 2) FF_LAUNCH(k_gemv_mfma<2>, grid, 256, 0, s, a);
    else FF_LAUNCH(k_gemv_mfma<4>, grid, 256, 0, s, a);
    return hipGetLastError();
  }
  // fp32: one launch per group of kGemvTileB samples (each reads the weights)
  const int grid = cdiv(a.Nout, 4 * kGemvRows);
  for (int b0 = 0; b0 < a.B; b0 += kGemvTileB) {
    GemvArgs p = a;
    p.B = min(kGemvTileB, a.B - b0);
    p.x = a.x + (size_t)b0 * a.ldx;
    p.y = a.y + (size_t)b0 * a.ldy;
    if (a.add) p.add = a.add + (size_t)b0 * a.ldadd;
    const size_t lds = (size_t)p.B * kGemvKC * sizeof(float);
    FF_LAUNCH(k_gemv<DT_F32>, grid, 256, lds, s, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t gemv_batch(int dtype, const GemvBatch& bt, hipStream_t s) {
  if (bt.njobs <= 0) return hipSuccess;
  if (bt.B < 1 || bt.B > kGemvMaxB) return hipErrorInvalidValue;
  int nmax = 0;
  for (int i = 0; i < bt.njobs; ++i) nmax = max(nmax, bt.job[i].Nout);
  if (dtype == DT_BF16) {
    if (bt.K % 8) return hipErrorInvalidValue;
    const dim3 grid(cdiv(nmax, 16), bt.njobs);
    const int ng = cdiv(bt.B, 8);
    if (ng == 1) FF_LAUNCH(k_gemv_mfma_batch<1>, grid, 256, 0, s, bt);
    else if (ng == 2) FF_LAUNCH(k_gemv_mfma_batch<2>, grid, 256, 0, s, bt);
    else FF_LAUNCH(k_gemv_mfma_batch<4>, grid, 256, 0, s, bt);
    return hipGetLastError();
  }
  const dim3 grid(cdiv(nmax, 4 * kGemvRows), bt.njobs);
  for (int b0 = 0; b0 < bt.B; b0 += kGemvTileB) {
    GemvBatch p = bt;
    p.B = min(kGemvTileB, bt.B - b0);
    p.x = bt.x + (size_t)b0 * bt.ldx;
    for (int i = 0; i < bt.njobs; ++i) p.job[i].y = bt.job[i].y + (size_t)b0 * bt.job[i].ldy;
    const size_t lds = (size_t)p.B * kGemvKC * sizeof(float);
    FF_LAUNCH(k_gemv_batch<DT_F32>, grid, 256, lds, s, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t time_embed(double sv, float* phi, hipStream_t st) {
  FF_LAUNCH(k_time_embed, 1, 128, 0, st, sv, phi);
  return hipGetLastError();
}

hipError_t time_embed_steps(double T, int n, float* phi, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  FF_LAUNCH(k_time_embed_steps, n, 128, 0, st, T, n, phi);
  return hipGetLastError();
}

hipError_t cond_split(const float* u, const float* cond, int nsteps, int B, int C, uint16_t* xs, float* cs,
                      uint16_t* zb, int nzb, hipStream_t st) {
  const long rows = xs ? (long)(B + 7) / 8 * 8 : B;
  const long tot = std::max((long)nsteps * rows * C, (long)nzb);
  if (tot <= 0) return hipSuccess;
  FF_LAUNCH(k_cond_split, cdiv(tot, 256), 256, 0, st, u, cond, nsteps, B, C, xs, cs, zb, nzb);
  return hipGetLastError();
}

hipError_t mod_combine(int dtype, const float* out, int N, const void* bias, float* dst, int ldy, int nb, int B,
                       hipStream_t st) {
  if (N % 4) return hipErrorInvalidValue;
  const long tot = (long)nb * B * (N / 4);
  if (tot <= 0) return hipSuccess;
  if (dtype == DT_BF16) FF_LAUNCH(k_mod_combine<DT_BF16>, cdiv(tot, 256), 256, 0, st, out, N, bias, dst, ldy, nb, B);
  else FF_LAUNCH(k_mod_combine<DT_F32>, cdiv(tot, 256), 256, 0, st, out, N, bias, dst, ldy, nb, B);
  return hipGetLastError();
}

hipError_t silu_rows(const float* x, float* y, int B, int n, uint16_t* xs, hipStream_t st) {
  if (xs && B > kGemvMaxB) return hipErrorInvalidValue;
  const long tot = (long)B * n;
  FF_LAUNCH(k_silu_rows, cdiv(tot, 256), 256, 0, st, x, y, B, n, xs);
  return hipGetLastError();
}

hipError_t patchify(int dtype, const float* x, void* patches, const PatchGeom& g, hipStream_t st) {
  const long n = (long)g.B * g.lat_c * g.F * g.H * g.W;
  if (dtype == DT_BF16) FF_LAUNCH(k_patchify<DT_BF16>, cdiv(n, 256), 256, 0, st, x, patches, g);
  else FF_LAUNCH(k_patchify<DT_F32>, cdiv(n, 256), 256, 0, st, x, patches, g);
  return hipGetLastError();
}

hipError_t unpatchify_euler(const float* yv, float* x, float dt, const PatchGeom& g, hipStream_t st) {
  const long n = (long)(g.lat_B ? g.lat_B : g.B) * g.lat_c * g.F * g.H * g.W;
  FF_LAUNCH(k_unpatchify_euler, cdiv(n, 256), 256, 0, st, yv, x, dt, g);
  return hipGetLastError();
}


// Token rows per workgroup of the MFMA final layer: 8 (256 workgroups for DiT-XL/2's 2048
// tokens, every CU busy) ran 10.2 us against 10.9 us for 16 (128 workgroups).
constexpr int kFinRows = 8;

// bf16 with at most 32 outputs per token and C <= kFinMfmaMaxC: the MFMA kernel
bool final_mfma(int dtype, int P, int C) {
  return dtype == DT_BF16 && P >= 1 && P <= 32 && C % 16 == 0 && C >= 16 && C <= kFinMfmaMaxC;
}

bool final_layer_ok(int dtype, int P, int C) {
  return final_mfma(dtype, P, C) ||
         ((P == 16 || P == 32 || P == 64) && C % 4 == 0 && C <= 4096 && (size_t)P * C * dsize(dtype) <= kFinalMaxWeightBytes);
}

hipError_t final_layer(int dtype, const FinalArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int P = a.g.pt * a.g.ph * a.g.pw * a.g.lat_c;
  if (!final_layer_ok(dtype, P, a.C)) return hipErrorInvalidValue;
  if (final_mfma(dtype, P, a.C)) {
    FF_LAUNCH(k_final_mfma<kFinRows>, cdiv(a.rows, kFinRows), 512, 0, s, a);
    return hipGetLastError();
  }
  const int grid = cdiv(a.rows, 4);
  const int units = cdiv(a.C / 4, 64);
#define FF_FIN(U, NP)                                                                   \
  do {                                                                                  \
    if (dtype == DT_BF16) FF_LAUNCH((k_final_layer<DT_BF16, U, NP>), grid, 256, 0, s, a); \
    else FF_LAUNCH((k_final_layer<DT_F32, U, NP>), grid, 256, 0, s, a);                 \
  } while (0)
#define FF_FIN_U(NP)                          \
  do {                                        \
    if (units <= 2) FF_FIN(2, NP);            \
    else if (units <= 5) FF_FIN(5, NP);       \
    else if (units <= 8) FF_FIN(8, NP);       \
    else if (units <= 12) FF_FIN(12, NP);     \
    else FF_FIN(16, NP);                      \
  } while (0)
  if (P == 16) FF_FIN_U(16);
  else if (P == 32) FF_FIN_U(32);
  else FF_FIN_U(64);
#undef FF_FIN_U
#undef FF_FIN
  return hipGetLastError();
}

}  // namespace ff
