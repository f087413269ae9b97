// Dense contractions of the exact block: out = epi(A W^T + bias) with A [M, K] (rows
// through a RowMap), W [N, K] (both K-contiguous), fp32 accumulation.
//
// bf16: v_mfma_f32_32x32x16_bf16 on 256x256 or 128x128 workgroup tiles, fed from LDS.
// The main kernel streams operands global -> LDS directly through a multi-stage ring; a
// register-staged kernel (padded LDS rows, double buffer) covers K % 32 != 0.
// fp32: 64x64x16 tile of plain FMAs (the small fp32 workload is launch-bound).
#include "dev_common.h"

namespace ff {

namespace {

// Template-only epilogue value: bias, plus GELU where the problem's own a.epi asks for it
// (a uniform branch per tile), so that a bias GEMM and a bias+GELU GEMM can share a launch.
constexpr int EPI_BIAS_OR_GELU = 3;


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

// Elements (uint16) of LDS the epilogue stages per workgroup: each wave owns 32 rows of
// its WN columns in fp32 (the worst case), rows padded by 4 floats.
template <int NW, int WN>
constexpr int epi_lds_elems() { return NW * 32 * (WN + 4) * 2; }

// Epilogue of one wavefront's TM x TN block of 32x32 MFMA tiles (acc), whose rows start at
// rbase and columns at cbase.  In the MFMA layout lane l owns row rbase + 32 i + l%32 and,
// per 32-column tile, 4 groups of 4 consecutive columns (8 q + 4 (l/32)): a store
// instruction there writes 8 bytes to each of 32 rows, which costs the memory pipeline one
// request per row.  So each 32-row block goes through the wave's own LDS region (lds):
// values are finished as far as the MFMA layout allows (bias, GELU) and staged as rows,
// as rounded bf16 when that is the output, else in fp32 (the gated residual is added to
// the unrounded value).  They are read back with consecutive lanes on consecutive
// 8-column pieces of a row, so every residual, gate and history load and every store is
// a 16-byte access and one instruction covers whole row segments.  The physical row (and
// sample) of each row is computed once by the lane that owns it in the MFMA layout and
// fetched by the storing lanes with a lane shuffle.  N % 8 == 0: a piece is in range as a
// whole.  LDS use is wave-private: the caller must have retired the main loop's LDS reads
// of all waves (barrier) before the first call.
template <int TM, int TN, int EPI, bool OUT_F32, bool RES_F32>
__device__ __forceinline__ void epilogue_block(const GemmArgs a, int rbase, int cbase, const f32x16_t (&acc)[TM][TN], uint16_t* lds) {
  constexpr bool kF32 = OUT_F32 || EPI == EPI_GATED;
  constexpr int WN = TN * 32, CPR = WN / 8, RPP = 64 / CPR, NPASS = (32 + RPP - 1) / RPP;
  constexpr int LDW = kF32 ? WN + 4 : WN + 8;   // row pitch in staged elements
  static_assert(CPR <= 64, "row wider than a wavefront's pieces");
  constexpr bool kCache = EPI == EPI_GATED && !OUT_F32;
  const int lane = threadIdx.x & 63, fr = lane & 31, fh = lane >> 5;
  const uint16_t* bias = reinterpret_cast<const uint16_t*>(a.bias);
  const bool gelu = EPI == EPI_BIAS_GELU || (EPI == EPI_BIAS_OR_GELU && a.epi == EPI_BIAS_GELU);
  float* lf = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int rmine = rbase + i * 32 + fr;
    const int prow = a.omap.phys(rmine < a.M ? rmine : 0);
    const int srow = EPI == EPI_GATED ? a.omap.sample(rmine < a.M ? rmine : 0) : 0;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = cbase + j * 32 + q * 8 + fh * 4;
        const u32x2_t bw = *reinterpret_cast<const u32x2_t*>(bias + (c < a.N ? c : 0));
        float v[4] = {acc[i][j][4 * q] + __uint_as_float(bw[0] << 16), acc[i][j][4 * q + 1] + __uint_as_float(bw[0] & 0xffff0000u),
                      acc[i][j][4 * q + 2] + __uint_as_float(bw[1] << 16), acc[i][j][4 * q + 3] + __uint_as_float(bw[1] & 0xffff0000u)};
        if (gelu) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = gelu_tanh_f(v[e]);
        }
        const int off = fr * LDW + j * 32 + q * 8 + fh * 4;
        if (kF32) {
          *reinterpret_cast<f32x4_t*>(lf + off) = f32x4_t{v[0], v[1], v[2], v[3]};
        } else {
          *reinterpret_cast<u32x2_t*>(lds + off) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        }
      }
    if (!kF32) {
#pragma unroll
      for (int p = 0; p < NPASS; ++p) {
        const int rr = p * RPP + lane / CPR, cc = (lane % CPR) * 8;
        const int src = rr < 32 ? rr : 0;
        const size_t pr = (size_t)__shfl(prow, src, 64);
        const int r = rbase + i * 32 + rr, c = cbase + cc;
        if (lane >= RPP * CPR || rr >= 32 || r >= a.M || c >= a.N) continue;
        *reinterpret_cast<u32x4_t*>(reinterpret_cast<uint16_t*>(a.out) + pr * a.ldo + c) =
            *reinterpret_cast<const u32x4_t*>(lds + rr * LDW + cc);
      }
      continue;
    }
    // fp32-staged rows, in groups of PG passes: every global load of a group (residual,
    // gate, and the layer input of the history refresh) is requested before the group's
    // first use.  Lanes that store nothing load row pr, column 0 (in range) and skip the
    // rest.  With the loads under the per-pass lane test, each pass waited for its own
    // loads (twice with the history refresh): up to 14 memory round trips per row block.
    constexpr int PG = NPASS < 4 ? NPASS : 4;
    const bool want_u = kCache && a.cache_out && a.cache_u;
#pragma unroll
    for (int p0 = 0; p0 < NPASS; p0 += PG) {
      size_t gpr[PG];
      int gc[PG], grr[PG], gcc[PG];
      bool ok[PG];
      f32x4_t rsf[PG][2], gg[PG][2];
      u32x4_t rsb[PG], uu[PG];
#pragma unroll
      for (int q = 0; q < PG; ++q) {
        const int p = p0 + q;
        if (p >= NPASS) break;
        const int rr = p * RPP + lane / CPR, cc = (lane % CPR) * 8;
        const int src = rr < 32 ? rr : 0;
        const size_t pr = (size_t)__shfl(prow, src, 64);
        const int sr = EPI == EPI_GATED ? __shfl(srow, src, 64) : 0;
        const int r = rbase + i * 32 + rr, c = cbase + cc;
        ok[q] = !(lane >= RPP * CPR || rr >= 32 || r >= a.M || c >= a.N);
        const int cl = ok[q] ? c : 0;
        gpr[q] = pr; gc[q] = c; grr[q] = rr; gcc[q] = cc;
        if (EPI == EPI_GATED) {
          if (RES_F32) {
            const float* rp = reinterpret_cast<const float*>(a.resid) + pr * a.ldr + cl;
            rsf[q][0] = *reinterpret_cast<const f32x4_t*>(rp);
            rsf[q][1] = *reinterpret_cast<const f32x4_t*>(rp + 4);
          } else {
            rsb[q] = *reinterpret_cast<const u32x4_t*>(reinterpret_cast<const uint16_t*>(a.resid) + pr * a.ldr + cl);
          }
          const float* gp = a.gate + (size_t)sr * a.ldg + cl;
          gg[q][0] = *reinterpret_cast<const f32x4_t*>(gp);
          gg[q][1] = *reinterpret_cast<const f32x4_t*>(gp + 4);
        }
        if (want_u) uu[q] = *reinterpret_cast<const u32x4_t*>(reinterpret_cast<const uint16_t*>(a.cache_u) + pr * a.ldo + cl);
      }
#pragma unroll
      for (int q = 0; q < PG; ++q) {
        if (p0 + q >= NPASS) break;
        if (!ok[q]) continue;
        const size_t pr = gpr[q];
        const int c = gc[q], rr = grr[q], cc = gcc[q];
        const f32x4_t x0 = *reinterpret_cast<const f32x4_t*>(lf + rr * LDW + cc);
        const f32x4_t x1 = *reinterpret_cast<const f32x4_t*>(lf + rr * LDW + cc + 4);
        float v[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        if (EPI == EPI_GATED) {
          float rs[8];
          if (RES_F32) {
#pragma unroll
            for (int e = 0; e < 4; ++e) { rs[e] = rsf[q][0][e]; rs[e + 4] = rsf[q][1][e]; }
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              rs[2 * e] = __uint_as_float(rsb[q][e] << 16);
              rs[2 * e + 1] = __uint_as_float(rsb[q][e] & 0xffff0000u);
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = rs[e] + gg[q][0][e] * v[e];
            v[e + 4] = rs[e + 4] + gg[q][1][e] * v[e + 4];
          }
        }
        if (OUT_F32) {
          St<DT_F32>::store(a.out, pr * a.ldo + c, v);
          St<DT_F32>::store(a.out, pr * a.ldo + c + 4, v + 4);
          continue;
        }
        St<DT_BF16>::store(a.out, pr * a.ldo + c, v);
        if (kCache && a.cache_out) {
          // history refresh from the stored (rounded) output, as the separate kernel does
          float h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) h[e] = St<DT_BF16>::rnd(v[e]);
          if (a.cache_u) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              h[2 * e] -= __uint_as_float(uu[q][e] << 16);
              h[2 * e + 1] -= __uint_as_float(uu[q][e] & 0xffff0000u);
            }
          }
          St<DT_BF16>::store(a.cache_out, pr * a.ldo + c, h);
        }
      }
    }
  }
}

// Up to two GEMMs of the same epilogue in one launch (the text and image streams of an
// MMDiT block): workgroups [0, n0) take problem 0's tiles, the rest problem 1's.
template <int NP>
struct GemmGroup {
  GemmArgs g[NP];
  int tm[NP], tn[NP];   // tile rows / columns per problem
};

// Workgroup -> (problem, output tile).  Workgroups are dispatched round-robin over the 8
// XCDs (each with its own L2); the first floor(n/8)*8 of them are renumbered so that every
// XCD owns a contiguous range of tiles, and within a problem tiles are ordered in groups
// of kGroupM tile-rows so that an XCD's concurrent tiles share A rows and W columns in its
// L2.
constexpr int kGroupM = 8;
__device__ __forceinline__ int tile_of(int bid, int tm0, int tn0, int tm1, int tn1, int np, int& tm, int& tn) {
  const int n0 = tm0 * tn0;
  const int nwg = n0 + (np > 1 ? tm1 * tn1 : 0);
  const int full = (nwg / 8) * 8;
  int id = bid < full ? (bid % 8) * (full / 8) + bid / 8 : bid;
  int p = 0, tiles_m = tm0, tiles_n = tn0;
  if (id >= n0) { p = 1; id -= n0; tiles_m = tm1; tiles_n = tn1; }
  const int per_group = kGroupM * tiles_n;
  const int first_m = (id / per_group) * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in_group = id % per_group;
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
  return p;
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
// Register-staged fallback (K % 32 != 0): BM x BN workgroup tile, BK = 64 per LDS stage
// with padded rows, wavefront tiles WM x WN of v_mfma_f32_32x32x16_bf16.
constexpr int BK = 64, LDT = BK + 8;

// 32x32x16 MFMA: A operand lane l = row (l%32), k 8*(l/32)..+7; B operand lane l = col (l%32),
// same k; D[v] at row 8*(v/4) + 4*(l/32) + v%4, col l%32.  With A = weight rows (output
// columns n) and B = activation rows (output rows m): lane l owns output row m = l%32 and
// columns n = 8*(v/4) + 4*(l/32) + (v%4), i.e. 4 groups of 4 consecutive columns.
template <int BM, int BN, int WM, int WN, int EPI, bool OUT_F32, bool RES_F32, int NP>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void k_gemm_bf16(GemmGroup<NP> G) {
  constexpr int NWN = BN / WN;
  constexpr int NT = (BM / WM) * NWN * 64;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int RSTEP = NT / 8;
  constexpr int CA = BM / RSTEP, CB = BN / RSTEP;
  constexpr int kMain = 2 * (BM + BN) * LDT, kEpi = epi_lds_elems<(BM / WM) * NWN, WN>();
  __shared__ __attribute__((aligned(1024))) uint16_t smem[kMain > kEpi ? kMain : kEpi];
  uint16_t (*sA)[BM * LDT] = reinterpret_cast<uint16_t (*)[BM * LDT]>(smem);
  uint16_t (*sB)[BN * LDT] = reinterpret_cast<uint16_t (*)[BN * LDT]>(smem + 2 * BM * LDT);
  // wave index in a scalar register: the per-wave LDS addresses of the DMA (M0) are then
  // computed on the scalar unit instead of with a v_readfirstlane per instruction
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  // workgroup-uniform: keep the problem select and tile origin in scalar registers
  const int prob = __builtin_amdgcn_readfirstlane(tile_of(blockIdx.x, G.tm[0], G.tn[0], G.tm[NP - 1], G.tn[NP - 1], NP, tm, tn));
  tm = __builtin_amdgcn_readfirstlane(tm);
  tn = __builtin_amdgcn_readfirstlane(tn);
  const GemmArgs a = (NP > 1 && prob) ? G.g[NP - 1] : G.g[0];
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
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  const int wm = (wave / NWN) * WM, wn = (wave % NWN) * WN;
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  const int nk = (a.K + BK - 1) / BK;
  FF_GLOAD(0);
  FF_SSTORE(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) FF_GLOAD((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t fa[TM], fb[TN];
#pragma unroll
      for (int t = 0; t < TM; ++t)
        fa[t] = *reinterpret_cast<const bf16x8_t*>(&sA[cur][(wm + t * 32 + fr) * LDT + kk + fk]);
#pragma unroll
      for (int t = 0; t < TN; ++t)
        fb[t] = *reinterpret_cast<const bf16x8_t*>(&sB[cur][(wn + t * 32 + fr) * LDT + kk + fk]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_iglp_opt(0);   // interleave the LDS fragment reads with the MFMAs
    }
    if (kt + 1 < nk) FF_SSTORE(cur ^ 1);
    __syncthreads();
  }
#undef FF_GLOAD
#undef FF_SSTORE
  // the loop ends with a barrier after every wave's last LDS read
  epilogue_block<TM, TN, EPI, OUT_F32, RES_F32>(a, m0 + wm, n0 + wn, acc, smem + wave * 32 * (WN + 4) * 2);
}
// ------------------------------------------------------------------ bf16 MFMA GEMM, direct-to-LDS
// For K % BKd == 0 (BKd = 32 or 64).  Operand tiles go global -> LDS with
// global_load_lds_dwordx4 (no VGPR staging, no ds_write), into an NST-stage ring of
// BKd-wide K slices issued NST-1 slices ahead.  Each DMA instruction fills 1 KB of LDS in
// lane order (16 rows x 64 bytes, or 8 rows x 128 bytes), so rows cannot be padded;
// instead lane l of a row loads a 16-byte chunk XOR-swizzled by the row ((l%4) ^
// ((row>>2)&3), or (l%8) ^ ((row>>1)&7)), which keeps the fragment reads free of bank
// conflicts: a 16-row group of a read spreads over all 64 banks.  (With 128-byte rows, even
// rows sit on banks 0-31 and odd rows on 32-63, so the 64-wide swizzle takes row/2; the
// first version used row&7, which put rows r and r+8 on the same banks.)
//
// Synchronisation is explicit: the compiler's barrier lowering waits for ALL outstanding
// loads (it cannot tell which stage a DMA targets), which would remove the prefetch.  So a
// stage boundary waits only for the next stage (s_waitcnt vmcnt(n) with the later stages
// still in flight) and then s_barrier, as one volatile asm that is also a compiler memory
// barrier.  Fragments are double-buffered in registers across the 16-wide k steps: the
// reads of the next step (ds_read_b128 asm) are in flight while the MFMAs of the current
// one run, each step waits with lgkmcnt(TM+TN) for the older reads only, and volatile "+v"
// asms tie the fragments to the MFMAs so that none is consumed before its wait.  The one
// barrier per stage sits between its last k step and the next stage's first.
//
// KG = 2 doubles the waves without growing the tile: waves w and w + NW accumulate the
// same output block, the first over k steps 0-1 of every 64-wide stage and the second
// over steps 2-3 (only the first issues the DMA; the second's vmcnt waits pass at once and
// the stage barrier orders it).  With two waves per SIMD, one wave's LDS reads and barrier
// waits hide behind the other's MFMAs.  After the loop the second k group hands its fp32
// sums to the first through LDS (a fixed order: group 0 + group 1), which runs the epilogue.
#define FF_AS1(p) ((const __attribute__((address_space(1))) void*)(p))
#define FF_AS3(p) ((__attribute__((address_space(3))) void*)(p))

// Wait until at most later * PER of this wave's DMA instructions are outstanding, then
// barrier.  A later beyond the cases waits for more than needed, which is safe.
template <int PER>
__device__ __forceinline__ void wait_stage(int later) {
  static_assert(3 * PER <= 63, "vmcnt field");
  switch (later) {
    case 0: asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(PER) : "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(2 * PER) : "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(3 * PER) : "memory"); break;
  }
}

__device__ __forceinline__ bf16x8_t lds_rd128(const uint16_t* p) {
  u32x4_t v;
  const uint32_t off = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) const void*)p);
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(off) : "memory");
  return __builtin_bit_cast(bf16x8_t, v);
}

template <int BM, int BN, int WM, int WN, int NST, int BKd, int KG, int AUX, int EPI, bool OUT_F32, bool RES_F32, int NP>
__global__ __launch_bounds__(KG * (BM / WM) * (BN / WN) * 64) void k_gemm_dl(GemmGroup<NP> G) {
  constexpr int NWN = BN / WN;
  constexpr int NW = (BM / WM) * NWN;                            // output blocks (waves per k group)
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int CH = BKd / 8, RPI = 64 / CH, KS = BKd / 16;   // chunks per row, rows per DMA, k steps
  constexpr int KPG = KS / KG;                                   // k steps per stage of one k group
  constexpr int IA = BM / RPI / NW, IB = BN / RPI / NW;        // DMA instructions per wave per stage
  static_assert(BKd == 32 || BKd == 64, "stage width");
  static_assert((KG == 1 || KG == 2) && KPG % 2 == 0, "k groups take an even number of k steps");
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "every tile row loaded by one DMA lane");
  static_assert(NST >= 3 && NST <= 5 && TM + TN <= 15, "unsupported tile");
  constexpr int kMain = NST * (BM + BN) * BKd, kEpi = epi_lds_elems<NW, WN>();
  constexpr int kRed = KG > 1 ? NW * TM * TN * 16 * 64 * 2 : 0;   // k group 1's partial sums (fp32)
  __shared__ __attribute__((aligned(1024))) uint16_t smem[kMain > kEpi + kRed ? kMain : kEpi + kRed];
  uint16_t (*sA)[BM * BKd] = reinterpret_cast<uint16_t (*)[BM * BKd]>(smem);
  uint16_t (*sB)[BN * BKd] = reinterpret_cast<uint16_t (*)[BN * BKd]>(smem + NST * BM * BKd);
  // wave index in a scalar register: the per-wave LDS addresses of the DMA (M0) are then
  // computed on the scalar unit instead of with a v_readfirstlane per instruction.  With
  // KG = 2, waves w and w + NW own the same output block (cw) and split every stage's k
  // steps between them (k group grp); only k group 0 issues the DMA.
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = KG > 1 ? wave / NW : 0, cw = KG > 1 ? wave % NW : wave;
  int tm, tn;
  // workgroup-uniform: keep the problem select and tile origin in scalar registers
  const int prob = __builtin_amdgcn_readfirstlane(tile_of(blockIdx.x, G.tm[0], G.tn[0], G.tm[NP - 1], G.tn[NP - 1], NP, tm, tn));
  tm = __builtin_amdgcn_readfirstlane(tm);
  tn = __builtin_amdgcn_readfirstlane(tn);
  const GemmArgs a = (NP > 1 && prob) ? G.g[NP - 1] : G.g[0];
  const int m0 = tm * BM, n0 = tn * BN;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(a.A);
  const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);
  auto swz = [](int ch, int row) { return BKd == 64 ? (ch ^ ((row >> 1) & 7)) : (ch ^ ((row >> 2) & 3)); };
  // rows past the matrix read row 0 (in bounds); their results are never stored
  const int lr = lane / CH, ls = lane % CH;
  size_t ga[IA], gb[IB];
#pragma unroll
  for (int j = 0; j < IA; ++j) {
    const int row = (cw * IA + j) * RPI + lr, gm = m0 + row;
    ga[j] = (size_t)a.amap.phys(gm < a.M ? gm : 0) * a.lda + swz(ls, row) * 8;
  }
#pragma unroll
  for (int j = 0; j < IB; ++j) {
    const int row = (cw * IB + j) * RPI + lr, gn = n0 + row;
    gb[j] = (size_t)(gn < a.N ? gn : 0) * a.ldw + swz(ls, row) * 8;
  }
#define FF_ISSUE(st, k0)                                                                                  \
  do {                                                                                                    \
    if (KG == 1 || grp == 0) {                                                                            \
      _Pragma("unroll") for (int j = 0; j < IA; ++j)                                                      \
        __builtin_amdgcn_global_load_lds(FF_AS1(A + ga[j] + (k0)), FF_AS3(&sA[st][(cw * IA + j) * RPI * BKd]), 16, 0, AUX); \
      _Pragma("unroll") for (int j = 0; j < IB; ++j)                                                      \
        __builtin_amdgcn_global_load_lds(FF_AS1(W + gb[j] + (k0)), FF_AS3(&sB[st][(cw * IB + j) * RPI * BKd]), 16, 0, AUX); \
    }                                                                                                     \
  } while (0)

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  const int wm = (cw / NWN) * WM, wn = (cw % NWN) * WN;
  const int fr = lane & 31, fh = lane >> 5;
  // fragment offsets within a stage for this k group's 16-wide k steps
  int offa[KPG][TM], offb[KPG][TN];
#pragma unroll
  for (int kk = 0; kk < KPG; ++kk) {
    const int ks = grp * KPG + kk;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      const int row = wm + t * 32 + fr;
      offa[kk][t] = row * BKd + swz(ks * 2 + fh, row) * 8;
    }
#pragma unroll
    for (int t = 0; t < TN; ++t) {
      const int row = wn + t * 32 + fr;
      offb[kk][t] = row * BKd + swz(ks * 2 + fh, row) * 8;
    }
  }
  const int nk = a.K / BKd;
#pragma unroll
  for (int s = 0; s < NST - 1; ++s)
    if (s < nk) FF_ISSUE(s, s * BKd);
  wait_stage<IA + IB>(min(NST - 2, nk - 1));   // stage 0 landed
  bf16x8_t fa[2][TM], fb[2][TN];
#pragma unroll
  for (int t = 0; t < TM; ++t) fa[0][t] = lds_rd128(&sA[0][offa[0][t]]);
#pragma unroll
  for (int t = 0; t < TN; ++t) fb[0][t] = lds_rd128(&sB[0][offb[0][t]]);
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt % NST;
#pragma unroll
    for (int s = 0; s < KPG; ++s) {
      const int cur = s & 1, nxt = cur ^ 1;   // KPG is even: stage k step 0 is always buffer 0
      if (s + 1 < KPG) {
#pragma unroll
        for (int t = 0; t < TM; ++t) fa[nxt][t] = lds_rd128(&sA[st][offa[s + 1][t]]);
#pragma unroll
        for (int t = 0; t < TN; ++t) fb[nxt][t] = lds_rd128(&sB[st][offb[s + 1][t]]);
        asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(TM + TN) : "memory");
      } else if (kt + 1 < nk) {
        // stage kt+1 complete everywhere, and every wave is past its reads of stage kt-1,
        // whose buffer now takes stage kt+NST-1; then the first k step of stage kt+1 is
        // read while the last one of stage kt computes
        wait_stage<IA + IB>(min(NST - 3, nk - 2 - kt));
        if (kt + NST - 1 < nk) FF_ISSUE((kt + NST - 1) % NST, (kt + NST - 1) * BKd);
        const int sn = (kt + 1) % NST;
#pragma unroll
        for (int t = 0; t < TM; ++t) fa[nxt][t] = lds_rd128(&sA[sn][offa[0][t]]);
#pragma unroll
        for (int t = 0; t < TN; ++t) fb[nxt][t] = lds_rd128(&sB[sn][offb[0][t]]);
        asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(TM + TN) : "memory");
      } else {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
#pragma unroll
      for (int t = 0; t < TM; ++t) asm volatile("" : "+v"(fa[cur][t]));
#pragma unroll
      for (int t = 0; t < TN; ++t) asm volatile("" : "+v"(fb[cur][t]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
    }
  }
#undef FF_ISSUE
  __syncthreads();   // every wave's last fragment reads retired before LDS is reused
  if (KG > 1) {
    // k group 1 hands its partial sums to k group 0 through LDS (past the epilogue staging)
    float* red = reinterpret_cast<float*>(smem + kEpi) + cw * TM * TN * 16 * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) red[((i * TN + j) * 16 + v) * 64] = acc[i][j][v];
    }
    __syncthreads();
    if (grp == 1) return;   // the epilogue has no workgroup barrier
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] += red[((i * TN + j) * 16 + v) * 64];
  }
  epilogue_block<TM, TN, EPI, OUT_F32, RES_F32>(a, m0 + wm, n0 + wn, acc, smem + cw * 32 * (WN + 4) * 2);
}

// ------------------------------------------------------------------ bf16 MFMA GEMM, 64-wide K stages
// For K % 64 == 0 on grids that keep the MFMAs busy for a whole stage (see launch_bf16).
// Two LDS buffers of 64-wide K stages: 128-byte rows (full cache lines per DMA row, 8 rows
// per 1 KB instruction), XOR swizzle chunk ^ ((row >> 1) & 7).  The DMA of stage kt+1 is issued
// right after the barrier that ends stage kt-1 (its buffer is free then) and lands during
// stage kt's four 16-wide k steps, whose fragments are double-buffered in registers as in
// k_gemm_dl; one wait + barrier per stage.
template <int BM, int BN, int WM, int WN, int AUX, int EPI, bool OUT_F32, bool RES_F32, int NP>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void k_gemm_dl64(GemmGroup<NP> G) {
  constexpr int BKd = 64, CH = 8, RPI = 8, KS = 4;
  constexpr int NWN = BN / WN;
  constexpr int NW = (BM / WM) * NWN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int IA = BM / RPI / NW, IB = BN / RPI / NW;
  static_assert(IA >= 1 && IB >= 1 && TM + TN <= 15, "unsupported tile");
  constexpr int kMain = 2 * (BM + BN) * BKd, kEpi = epi_lds_elems<NW, WN>();
  __shared__ __attribute__((aligned(1024))) uint16_t smem[kMain > kEpi ? kMain : kEpi];
  uint16_t (*sA)[BM * BKd] = reinterpret_cast<uint16_t (*)[BM * BKd]>(smem);
  uint16_t (*sB)[BN * BKd] = reinterpret_cast<uint16_t (*)[BN * BKd]>(smem + 2 * BM * BKd);
  // wave index in a scalar register: the per-wave LDS addresses of the DMA (M0) are then
  // computed on the scalar unit instead of with a v_readfirstlane per instruction
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int tm, tn;
  // workgroup-uniform: keep the problem select and tile origin in scalar registers
  const int prob = __builtin_amdgcn_readfirstlane(tile_of(blockIdx.x, G.tm[0], G.tn[0], G.tm[NP - 1], G.tn[NP - 1], NP, tm, tn));
  tm = __builtin_amdgcn_readfirstlane(tm);
  tn = __builtin_amdgcn_readfirstlane(tn);
  const GemmArgs a = (NP > 1 && prob) ? G.g[NP - 1] : G.g[0];
  const int m0 = tm * BM, n0 = tn * BN;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(a.A);
  const uint16_t* W = reinterpret_cast<const uint16_t*>(a.W);
  const int lr = lane / CH, ls = lane % CH;
  // Only waves 0..NW/2-1 issue the DMA, each for its own rows and those of wave + NW/2 (one
  // issuing wave per SIMD).  A stage's DMA goes out as a burst that can fill the L1's
  // outstanding-request queue; a wave stalled issuing it cannot issue its MFMAs either,
  // and with half the waves free of DMA every SIMD keeps a wave that can (DiT-XL/2 fc1
  // 35.0 -> 32.8 us, FLUX-like qkv, proj, fc2 and lin2 3-7 % faster).
  constexpr int HW = NW / 2;
  static_assert(NW % 2 == 0, "issuing waves pair with the upper half");
  size_t ga[2 * IA], gb[2 * IB];
  int wa[2 * IA], wb[2 * IB];
#pragma unroll
  for (int j = 0; j < 2 * IA; ++j) {
    const int w = j < IA ? wave : wave + HW, jj = j % IA;
    wa[j] = (w * IA + jj) * RPI * BKd;
    const int row = (w * IA + jj) * RPI + lr, gm = m0 + row;
    ga[j] = (size_t)a.amap.phys(gm < a.M ? gm : 0) * a.lda + ((ls ^ ((row >> 1) & 7)) * 8);
  }
#pragma unroll
  for (int j = 0; j < 2 * IB; ++j) {
    const int w = j < IB ? wave : wave + HW, jj = j % IB;
    wb[j] = (w * IB + jj) * RPI * BKd;
    const int row = (w * IB + jj) * RPI + lr, gn = n0 + row;
    gb[j] = (size_t)(gn < a.N ? gn : 0) * a.ldw + ((ls ^ ((row >> 1) & 7)) * 8);
  }
#define FF_ISSUE(st, k0)                                                                                  \
  do {                                                                                                    \
    if (wave < HW) {                                                                                      \
    _Pragma("unroll") for (int j = 0; j < 2 * IA; ++j)                                                    \
      __builtin_amdgcn_global_load_lds(FF_AS1(A + ga[j] + (k0)), FF_AS3(&sA[st][wa[j]]), 16, 0, AUX); \
    _Pragma("unroll") for (int j = 0; j < 2 * IB; ++j)                                                    \
      __builtin_amdgcn_global_load_lds(FF_AS1(W + gb[j] + (k0)), FF_AS3(&sB[st][wb[j]]), 16, 0, AUX); \
    }                                                                                                     \
  } while (0)
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  const int wm = (wave / NWN) * WM, wn = (wave % NWN) * WN;
  const int fr = lane & 31, fh = lane >> 5;
  int rowa[TM], rowb[TN];
#pragma unroll
  for (int t = 0; t < TM; ++t) rowa[t] = wm + t * 32 + fr;
#pragma unroll
  for (int t = 0; t < TN; ++t) rowb[t] = wn + t * 32 + fr;
  const int nk = a.K / BKd;
  FF_ISSUE(0, 0);
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  bf16x8_t fa[2][TM], fb[2][TN];
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) FF_ISSUE(st ^ 1, (kt + 1) * BKd);   // buffer of stage kt-1: free after the last barrier
#pragma unroll
    for (int t = 0; t < TM; ++t) fa[0][t] = lds_rd128(&sA[st][rowa[t] * BKd + ((fh ^ ((rowa[t] >> 1) & 7)) * 8)]);
#pragma unroll
    for (int t = 0; t < TN; ++t) fb[0][t] = lds_rd128(&sB[st][rowb[t] * BKd + ((fh ^ ((rowb[t] >> 1) & 7)) * 8)]);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int cur = s & 1, nxt = cur ^ 1;
      if (s + 1 < KS) {
        const int ch = (s + 1) * 2 + fh;
#pragma unroll
        for (int t = 0; t < TM; ++t) fa[nxt][t] = lds_rd128(&sA[st][rowa[t] * BKd + ((ch ^ ((rowa[t] >> 1) & 7)) * 8)]);
#pragma unroll
        for (int t = 0; t < TN; ++t) fb[nxt][t] = lds_rd128(&sB[st][rowb[t] * BKd + ((ch ^ ((rowb[t] >> 1) & 7)) * 8)]);
        asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(TM + TN) : "memory");
      } else {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
#pragma unroll
      for (int t = 0; t < TM; ++t) asm volatile("" : "+v"(fa[cur][t]));
#pragma unroll
      for (int t = 0; t < TN; ++t) asm volatile("" : "+v"(fb[cur][t]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
    }
    // stage kt+1 landed everywhere, and every wave is done reading stage kt.  The
    // scheduling fence keeps every MFMA of this stage above the wait: the compiler would
    // otherwise sink them below the barrier (they touch no memory), which delays the next
    // stage's DMA by their issue time and idles the matrix cores during the wait
    // (FLUX-like qkv 293 -> 264 us, DiT-XL/2 fc1 39.3 -> 36.4 us)
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  }
#undef FF_ISSUE
  // the loop ends with a barrier after every wave's last LDS read
  epilogue_block<TM, TN, EPI, OUT_F32, RES_F32>(a, m0 + wm, n0 + wn, acc, smem + wave * 32 * (WN + 4) * 2);
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

template <int BM, int BN, int NP>
GemmGroup<NP> make_group(const GemmArgs* a, int& nwg) {
  GemmGroup<NP> G{};
  nwg = 0;
  for (int i = 0; i < NP; ++i) {
    G.g[i] = a[i];
    G.tm[i] = (a[i].M + BM - 1) / BM;
    G.tn[i] = (a[i].N + BN - 1) / BN;
    nwg += G.tm[i] * G.tn[i];
  }
  return G;
}

template <int BM, int BN, int WM, int WN, int EPI, bool OF, bool RF>
void launch_tile(const GemmArgs* a, int n, hipStream_t s) {
  int nwg;
  if (n == 1) {
    const GemmGroup<1> G = make_group<BM, BN, 1>(a, nwg);
    FF_LAUNCH((k_gemm_bf16<BM, BN, WM, WN, EPI, OF, RF, 1>), nwg, (BM / WM) * (BN / WN) * 64, 0, s, G);
  } else {
    const GemmGroup<2> G = make_group<BM, BN, 2>(a, nwg);
    FF_LAUNCH((k_gemm_bf16<BM, BN, WM, WN, EPI, OF, RF, 2>), nwg, (BM / WM) * (BN / WN) * 64, 0, s, G);
  }
}

template <int BM, int BN, int WM, int WN, int NST, int BKd, int KG, int AUX, int EPI, bool OF, bool RF>
void launch_dl(const GemmArgs* a, int n, hipStream_t s) {
  int nwg;
  if (n == 1) {
    const GemmGroup<1> G = make_group<BM, BN, 1>(a, nwg);
    FF_LAUNCH((k_gemm_dl<BM, BN, WM, WN, NST, BKd, KG, AUX, EPI, OF, RF, 1>), nwg, KG * (BM / WM) * (BN / WN) * 64, 0, s, G);
  } else {
    const GemmGroup<2> G = make_group<BM, BN, 2>(a, nwg);
    FF_LAUNCH((k_gemm_dl<BM, BN, WM, WN, NST, BKd, KG, AUX, EPI, OF, RF, 2>), nwg, KG * (BM / WM) * (BN / WN) * 64, 0, s, G);
  }
}

template <int BM, int BN, int WM, int WN, int AUX, int EPI, bool OF, bool RF>
void launch_dl64(const GemmArgs* a, int n, hipStream_t s) {
  int nwg;
  if (n == 1) {
    const GemmGroup<1> G = make_group<BM, BN, 1>(a, nwg);
    FF_LAUNCH((k_gemm_dl64<BM, BN, WM, WN, AUX, EPI, OF, RF, 1>), nwg, (BM / WM) * (BN / WN) * 64, 0, s, G);
  } else {
    const GemmGroup<2> G = make_group<BM, BN, 2>(a, nwg);
    FF_LAUNCH((k_gemm_dl64<BM, BN, WM, WN, AUX, EPI, OF, RF, 2>), nwg, (BM / WM) * (BN / WN) * 64, 0, s, G);
  }
}

// Tile choice for K % 64 == 0: the candidate minimising (rounds of workgroups over the
// 256 CUs) x (time of one round of that candidate), measured on MI355X with random bf16
// data and expressed relative to a round of 256x256 tiles (the ratio drifts with K, e.g.
// 0.36 at K = 1152 and 0.29 at K = 4608 for 128x96; the constants sit between).
//   kTile256     256x256, 8 waves of 128x64, 2 x 64-wide stages, 1 per CU          1.00
//   kTile256x192 256x192, 8 waves of 64x96,  2 x 64-wide stages, 1 per CU          0.91
//   kTile128x2   128x128, 8 waves of 64x32, 2 x 64-wide stages, 2 per CU (512/round) 0.80
//   kTile128     128x128, 4 blocks of 64x64 x 2 k groups, 4 x 64-wide stages        0.41
//   kTile128x96  128x96,  4 blocks of 32x96 x 2 k groups, 4 x 64-wide stages        0.34
//   kTile128x64  128x64,  4 blocks of 32x64 x 2 k groups, 4 x 64-wide stages        0.24
// Larger tiles need fewer operand bytes per MFMA (LDS traffic per MFMA limits the 128x128
// tiles), smaller ones fill the CUs on small grids (M = 2048 shapes).  The 128-row ring
// tiles run two k groups of waves per output block (8 waves, two per SIMD): one wave's
// LDS reads and barrier waits then overlap the other's MFMAs.  Operands of the 256-row
// tiles load with sc0|sc1 (they skip the L1; each tile streams its panels once).
// A group is costed by its total tile count.  K % 32 == 0 only: 4 x 32-wide stages,
// 256x256 from 160 such tiles on, else 128x128; otherwise the register-staged kernel.
enum { kTile256, kTile256x192, kTile128x2, kTile128, kTile128x96, kTile128x64, kTileCount };
struct TilePlan { int tile; double cost; };

long tiles_of(const GemmArgs* a, int n, int bm, int bn) {
  long t = 0;
  for (int i = 0; i < n; ++i) t += (long)((a[i].M + bm - 1) / bm) * ((a[i].N + bn - 1) / bn);
  return t;
}

TilePlan plan_k64(const GemmArgs* a, int n) {
  static const double kRound[kTileCount] = {1.00, 0.91, 0.80, 0.41, 0.34, 0.24};
  const long t[kTileCount] = {tiles_of(a, n, 256, 256), tiles_of(a, n, 256, 192), tiles_of(a, n, 128, 128),
                              tiles_of(a, n, 128, 128), tiles_of(a, n, 128, 96), tiles_of(a, n, 128, 64)};
  const long per_round[kTileCount] = {256, 256, 512, 256, 256, 256};
  TilePlan best{kTile256, 1e300};
  for (int c = 0; c < kTileCount; ++c) {
    const double cost = (double)((t[c] + per_round[c] - 1) / per_round[c]) * kRound[c];
    if (cost < best.cost) best = TilePlan{c, cost};
  }
  return best;
}

bool all_k(const GemmArgs* a, int n, int m) {
  for (int i = 0; i < n; ++i)
    if (a[i].K % m) return false;
  return true;
}

template <int EPI, bool OF, bool RF>
void launch_bf16(const GemmArgs* a, int n, hipStream_t s) {
  if (!all_k(a, n, 32)) {
    launch_tile<128, 128, 64, 32, EPI, OF, RF>(a, n, s);
  } else if (!all_k(a, n, 64)) {
    if (tiles_of(a, n, 256, 256) >= 160) launch_dl<256, 256, 128, 64, 4, 32, 1, 17, EPI, OF, RF>(a, n, s);
    else launch_dl<128, 128, 64, 32, 4, 32, 1, 0, EPI, OF, RF>(a, n, s);
  } else {
    switch (plan_k64(a, n).tile) {
      case kTile256: launch_dl64<256, 256, 128, 64, 17, EPI, OF, RF>(a, n, s); break;
      case kTile256x192: launch_dl64<256, 192, 64, 96, 17, EPI, OF, RF>(a, n, s); break;
      case kTile128x2: launch_dl64<128, 128, 64, 32, 0, EPI, OF, RF>(a, n, s); break;
      case kTile128: launch_dl<128, 128, 64, 64, 4, 64, 2, 17, EPI, OF, RF>(a, n, s); break;
      case kTile128x96: launch_dl<128, 96, 32, 96, 4, 64, 2, 17, EPI, OF, RF>(a, n, s); break;
      default: launch_dl<128, 64, 32, 64, 4, 64, 2, 0, EPI, OF, RF>(a, n, s); break;
    }
  }
}

}  // namespace

namespace {

// bf16 dispatch of n (1 or 2) problems that share epilogue, output and residual types
hipError_t gemm_bf16(const GemmArgs* a, int n, hipStream_t s) {
  const bool of = a[0].out_f32 != 0, rf = a[0].resid_f32 != 0;
  if (n == 2 && a[0].epi != a[1].epi) {   // bias with bias+GELU (gemm2 admits no other mix)
    if (of) launch_bf16<EPI_BIAS_OR_GELU, true, false>(a, n, s);
    else launch_bf16<EPI_BIAS_OR_GELU, false, false>(a, n, s);
    return hipGetLastError();
  }
  switch (a[0].epi) {
    case EPI_BIAS:
      if (of) launch_bf16<EPI_BIAS, true, false>(a, n, s);
      else launch_bf16<EPI_BIAS, false, false>(a, n, s);
      break;
    case EPI_BIAS_GELU:
      if (of) launch_bf16<EPI_BIAS_GELU, true, false>(a, n, s);
      else launch_bf16<EPI_BIAS_GELU, false, false>(a, n, s);
      break;
    default:
      if (of && rf) launch_bf16<EPI_GATED, true, true>(a, n, s);
      else if (of) launch_bf16<EPI_GATED, true, false>(a, n, s);
      else if (rf) launch_bf16<EPI_GATED, false, true>(a, n, s);
      else launch_bf16<EPI_GATED, false, false>(a, n, s);
      break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (dtype == DT_F32) {
    const int grid = ((a.M + 63) / 64) * ((a.N + 63) / 64);
    switch (a.epi) {
      case EPI_BIAS: FF_LAUNCH(k_gemm_f32<EPI_BIAS>, grid, 256, 0, s, a); break;
      case EPI_BIAS_GELU: FF_LAUNCH(k_gemm_f32<EPI_BIAS_GELU>, grid, 256, 0, s, a); break;
      default: FF_LAUNCH(k_gemm_f32<EPI_GATED>, grid, 256, 0, s, a); break;
    }
    return hipGetLastError();
  }
  return gemm_bf16(&a, 1, s);
}

hipError_t gemm2(int dtype, const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
  const bool e0 = a0.M > 0 && a0.N > 0, e1 = a1.M > 0 && a1.N > 0;
  const bool ungated = a0.epi != EPI_GATED && a1.epi != EPI_GATED;
  const bool same = (a0.epi == a1.epi || ungated) && a0.out_f32 == a1.out_f32 && a0.resid_f32 == a1.resid_f32;
  // Grouping pays when the combined launch costs no more rounds than the two launches
  // (same cost model as the tile choice; with K % 64 != 0, by 256x256 rounds).
  const GemmArgs both[2] = {a0, a1};
  bool pays;
  if (all_k(both, 2, 64)) {
    pays = plan_k64(both, 2).cost <= plan_k64(&a0, 1).cost + plan_k64(&a1, 1).cost;
  } else {
    const long t0 = tiles_of(&a0, 1, 256, 256), t1 = tiles_of(&a1, 1, 256, 256);
    const long rg = (t0 + t1 + 255) / 256, r0 = (t0 + 255) / 256, r1 = (t1 + 255) / 256;
    pays = t0 + t1 < 160 || rg <= (r0 > r1 ? r0 : r1) || ((t0 < t1 ? t0 : t1) >= 160 && rg < r0 + r1);
  }
  if (dtype == DT_F32 || !same || !e0 || !e1 || !pays) {
    hipError_t e = gemm(dtype, a0, s);
    return e != hipSuccess ? e : gemm(dtype, a1, s);
  }
  return gemm_bf16(both, 2, s);
}

}  // namespace ff
