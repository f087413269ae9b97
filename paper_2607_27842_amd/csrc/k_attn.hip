// Softmax attention softmax(q k^T * scale) v per (sample, head), flash-style: key/value
// tiles are staged through LDS and each wavefront keeps a running (max, sum) per query
// (online softmax), so no N x N matrix is ever stored.
//
// bf16: v_mfma_f32_32x32x16_bf16 (the full-rate gfx950 bf16 MFMA).  A wavefront owns 32
// queries; a workgroup of 4 or 8 wavefronts shares each 64-key tile.  Scores are formed
// transposed, S^T = K Q^T, so every lane holds the scores of ONE query: the softmax
// statistics are lane-local plus one cross-lane step, and the probabilities are already
// in the register layout of the B operand of O^T = V^T P^T (no shuffle).
// fp32: one thread per query, 32-key LDS tiles (small fp32 workloads only).
#include "dev_common.h"

namespace ff {

namespace {

constexpr int KT = 64;  // keys per LDS tile
constexpr float kLazy = 8.0f;  // log2 headroom before the running max is raised

// ---------------------------------------------------------------- bf16, 32x32x16 MFMA
// NW wavefronts x 32 queries per workgroup; 64-key K/V tiles staged through LDS (K row-
// major, V transposed), the next tile prefetched into registers during the current one.
// v_mfma_f32_32x32x16_bf16 layouts (A lane l: row l%32, k 8*(l/32)+0..7; B lane l: col
// l%32, same k; D[v] at row 8*(v/4) + 4*(l/32) + v%4, col l%32):
//   S^T = K Q^T : A = K (32 keys x 16 dims), B = Q^T (16 dims x 32 queries) -> lane l holds
//                 16 scores of query l%32, keys 8*(v/4) + 4*(l/32) + v%4 of a 32-key tile.
//   O^T += V^T P^T : B = P^T needs, per lane, the probabilities of query l%32 at 8 keys
//                 for the MFMA k index 8*(l/32)+j; mapping k index j to key
//                 (j<4 ? 4h+j : 8+4h+j-4) (+16 for the second half of the tile) makes that
//                 exactly the registers the lane already holds.  A = V^T rows (e) at those
//                 keys; the transposed V tile stores key k of each 16-key group at column
//                 vpos(k) (bits 2 and 3 swapped), which makes them one 16-byte LDS read.
// Head dims are zero-padded: QK^T to a multiple of 16 (DQ), PV to a multiple of 32 (DV).
__device__ __forceinline__ int vpos(int k) { return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1); }

// The two halves of a wavefront exchanged in registers (v_permlane32_swap, no LDS round
// trip): every lane gets lo = x of lane l % 32 and hi = x of lane l % 32 + 32, so a
// combination of lo and hi is the same value in lanes l and l ^ 32.
__device__ __forceinline__ void wave_halves(float x, float& lo, float& hi) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  lo = __uint_as_float(r[0]);
  hi = __uint_as_float(r[1]);
}

template <int DQ, int DV, int NW, int SPLIT, int KTL>   // KTL: keys per LDS tile (64 or 128)
__global__ __launch_bounds__(NW * SPLIT * 64) void k_attn32(AttnArgs a) {
  constexpr int NS = KTL / 32;        // 32-key score tiles per LDS tile
  constexpr int NT = NW * 64;   // threads of one group
  constexpr int LDK = DQ + 8;         // K tile row stride (elements)
  constexpr int LDV = KTL + 8;        // V^T tile row stride
  constexpr int NQC = DQ / 16;        // 16-wide head-dim chunks of QK^T
  constexpr int NOT = DV / 32;        // 32-wide output tiles of the head dim
  constexpr int KCH = KTL * (DQ / 8); // 16-byte chunks of a K tile
  constexpr int PK = (KCH + NT - 1) / NT;
  constexpr int VG = (KTL / 4) * (DV / 8);  // V groups: 4 consecutive keys x 8 head dims
  constexpr int PV = (VG + NT - 1) / NT;
  static_assert(DV <= DQ + 16, "layout");
  // per group: two K tiles [KTL][LDK] and two V^T tiles [DV][LDV]
  constexpr int KSZ = KTL * LDK, VSZ = DV * LDV;
  __shared__ __attribute__((aligned(16))) uint16_t smem[SPLIT * 2 * (KSZ + VSZ)];
  auto Ks = [&](int g, int b) { return smem + (g * 2 + b) * KSZ; };
  auto Vt = [&](int g, int b) { return smem + SPLIT * 2 * KSZ + (g * 2 + b) * VSZ; };

  // SPLIT groups of NW wavefronts take the same queries over disjoint key ranges
  // a group is whole wavefronts (NT % 64 == 0): grp in a scalar register keeps the key tile
  // origin, and with it the tile base address and the in-range test, scalar
  const int grp = __builtin_amdgcn_readfirstlane(threadIdx.x / NT), gtid = threadIdx.x % NT;
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) % NW;
  const int c32 = lane & 31, h = lane >> 5;
  // Workgroups go to the 8 XCDs (each with its own L2) round-robin in launch order; the
  // first floor(n/8)*8 are renumbered so that each XCD takes a contiguous range of
  // (sample, head, query block) triples, query blocks fastest: the query blocks of one
  // head then read its K/V tiles through one L2 instead of all eight.
  int qb, hd, b;
  {
    const int nqb = (a.N + NW * 32 - 1) / (NW * 32), n = gridDim.x, id = blockIdx.x;
    const int full = n / 8 * 8;
    const int t = id < full ? (id % 8) * (full / 8) + id / 8 : id;
    qb = __builtin_amdgcn_readfirstlane(t % nqb);
    hd = __builtin_amdgcn_readfirstlane((t / nqb) % a.H);
    b = __builtin_amdgcn_readfirstlane(t / (nqb * a.H));
  }
  const int q0 = qb * (NW * 32) + wave * 32;
  const int N = a.N, d = a.d;
  const uint16_t* qkv = reinterpret_cast<const uint16_t*>(a.qkv);
  const size_t rb = (size_t)b * N;
  const size_t qoff = (size_t)hd * d, koff = (size_t)a.C + hd * d, voff = 2 * (size_t)a.C + hd * d;
  const u32x4_t z4 = {0u, 0u, 0u, 0u};

  // Q^T fragments: lane holds Q[q0 + c32][16c + 8h .. +7]
  bf16x8_t qf[NQC];
  {
    const int q = q0 + c32;
#pragma unroll
    for (int c = 0; c < NQC; ++c) {
      const int e = 16 * c + 8 * h;
      const u32x4_t v = (q < N && e < d) ? *reinterpret_cast<const u32x4_t*>(qkv + (rb + q) * a.ldq + qoff + e) : z4;
      qf[c] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
  f32x16_t o[NOT];
#pragma unroll
  for (int t = 0; t < NOT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[t][v] = 0.f;
  float mrow = -INFINITY, lrow = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;

  // Register prefetch of one K/V tile.  K: chunk c -> key c / (DQ/8), dims (c % (DQ/8))*8.
  // V: group g -> keys 4 (g % (KTL/4)) + 0..3, dims (g / (KTL/4))*8: each transposed row piece
  // (4 keys of one dim) is one 8-byte LDS store, and the 16 consecutive lanes of a store
  // fill one 128-byte V^T row segment (no bank conflicts).
  // Each load is a uniform 64-bit tile base (the tile's first key row) plus this lane's
  // 32-bit byte offset, fixed before the loop, so the per-tile address work is scalar and the
  // loads take the scalar-base form.  Tiles whose chunks are all in range (every key below
  // N, d equal to the padded head dims, every chunk owned) load without lane masks.
  u32x4_t pk[PK], pv[PV][4];
  uint32_t kbo[PK], vbo[PV];
  int kkr[PK], vk4[PV];
  bool kok[PK], vok[PV];
  const size_t rowb = (size_t)a.ldq * 2;   // bytes per token row of qkv
#pragma unroll
  for (int i = 0; i < PK; ++i) {
    const int c = gtid + i * NT;
    const int kr = c / (DQ / 8), e = (c % (DQ / 8)) * 8;
    kkr[i] = kr;
    kok[i] = c < KCH && e < d;
    kbo[i] = kok[i] ? (uint32_t)(kr * rowb + (koff + e) * 2) : 0u;
  }
#pragma unroll
  for (int i = 0; i < PV; ++i) {
    const int g = gtid + i * NT;
    const int k4 = (g % (KTL / 4)) * 4, e = (g / (KTL / 4)) * 8;
    vk4[i] = k4;
    vok[i] = g < VG && e < d;
    vbo[i] = vok[i] ? (uint32_t)(k4 * rowb + (voff + e) * 2) : 0u;
  }
  const bool dense_dims = d == DQ && d == DV && KCH % NT == 0 && VG % NT == 0;
  auto fetch = [&](int kv0) {
    const char* tb = reinterpret_cast<const char*>(qkv + (rb + kv0) * a.ldq);
    auto ld = [&](uint32_t off) { return *reinterpret_cast<const u32x4_t*>(tb + off); };
    if (dense_dims && kv0 + KTL <= N) {
#pragma unroll
      for (int i = 0; i < PK; ++i) pk[i] = ld(kbo[i]);
#pragma unroll
      for (int i = 0; i < PV; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) pv[i][r] = ld(vbo[i] + (uint32_t)(r * rowb));
    } else {
      const int lim = N - kv0;   // keys at or past it are masked
#pragma unroll
      for (int i = 0; i < PK; ++i) pk[i] = (kok[i] && kkr[i] < lim) ? ld(kbo[i]) : z4;
#pragma unroll
      for (int i = 0; i < PV; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) pv[i][r] = (vok[i] && vk4[i] + r < lim) ? ld(vbo[i] + (uint32_t)(r * rowb)) : z4;
    }
  };
  auto stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PK; ++i) {
      const int c = gtid + i * NT;
      if (c < KCH) {
        const int kr = c / (DQ / 8), e = (c % (DQ / 8)) * 8;
        *reinterpret_cast<u32x4_t*>(Ks(grp, buf) + kr * LDK + e) = pk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < PV; ++i) {
      const int g = gtid + i * NT;
      if (g < VG) {
        const int k4 = (g % (KTL / 4)) * 4, e = (g / (KTL / 4)) * 8;
        uint16_t* dst = Vt(grp, buf) + e * LDV + vpos(k4);   // keys k4..k4+3 stay consecutive under vpos
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          u32x2_t lo, hi;   // dims e + 2j and e + 2j + 1 of the four keys
          lo[0] = (pv[i][0][j] & 0xffffu) | (pv[i][1][j] << 16);
          lo[1] = (pv[i][2][j] & 0xffffu) | (pv[i][3][j] << 16);
          hi[0] = (pv[i][0][j] >> 16) | (pv[i][1][j] & 0xffff0000u);
          hi[1] = (pv[i][2][j] >> 16) | (pv[i][3][j] & 0xffff0000u);
          *reinterpret_cast<u32x2_t*>(dst + (2 * j) * LDV) = lo;
          *reinterpret_cast<u32x2_t*>(dst + (2 * j + 1) * LDV) = hi;
        }
      }
    }
  };
  // LDS writes done, then barrier; the global prefetch of the tile after next stays in flight
  // (the compiler's barrier would also wait for it)
#define FF_LDS_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")
  // this group's tiles: [t0, t0 + nt) of the ntiles key tiles (every group runs the same
  // number of iterations, so the workgroup barriers line up; a group past the end has
  // kv0 >= N, all its keys masked, and contributes nothing)
  const int ntiles = (N + KTL - 1) / KTL;
  const int nt = (ntiles + SPLIT - 1) / SPLIT, t0 = grp * nt;
  fetch(t0 * KTL);
  stage(0);
  if (nt > 1) fetch((t0 + 1) * KTL);
  FF_LDS_BARRIER();
  for (int kt = 0; kt < nt; ++kt) {
    const int kv0 = (t0 + kt) * KTL, buf = kt & 1;
    const uint16_t* K_ = Ks(grp, buf);
    const uint16_t* V_ = Vt(grp, buf);
    // scores for NS 32-key tiles
    f32x16_t sc[NS];
#pragma unroll
    for (int t = 0; t < NS; ++t) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[t][v] = 0.f;
#pragma unroll
      for (int c = 0; c < NQC; ++c) {
        const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(&K_[(t * 32 + c32) * LDK + 16 * c + 8 * h]);
        sc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[c], sc[t], 0, 0, 0);
      }
    }
    // online softmax for query q0 + c32 (its KTL scores: half in this lane, half in lane ^ 32).
    // The running max m is kept in log2 units of the scaled scores; it is raised (and O, l
    // rescaled) only when the tile's max exceeds it by more than kLazy, so most tiles skip
    // the rescale.  The shift cancels in O / l, and p <= 2^kLazy stays well inside fp32.
    float mx = -INFINITY;
    if (kv0 + KTL > N) {   // last, partial tile: keys past N get probability 0
#pragma unroll
      for (int t = 0; t < NS; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kv0 + 32 * t + 8 * (v >> 2) + 4 * h + (v & 3);
          if (key >= N) sc[t][v] = -INFINITY;
        }
    }
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[t][v]);
    {
      float lo, hi;
      wave_halves(mx, lo, hi);
      mx = fmaxf(lo, hi) * sl2;   // scale > 0: max commutes with it
    }
    if (mx > mrow + kLazy) {
      const float alpha = __builtin_amdgcn_exp2f(mrow - mx);   // v_exp_f32: exp2(-inf) = 0
      lrow *= alpha;
#pragma unroll
      for (int t = 0; t < NOT; ++t) o[t] *= alpha;
      mrow = mx;
    }
    // mrow is still -inf only if every score so far is -inf (all keys masked, as for a
    // group whose keys start past N): those probabilities are exp2(-inf) = 0, not NaN
    const float moff = mrow == -INFINITY ? 0.f : mrow;
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < NS; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float pr = __builtin_amdgcn_exp2f(fmaf(sc[t][v], sl2, -moff));
        sc[t][v] = pr;
        ls += pr;
      }
    {
      float lo, hi;
      wave_halves(ls, lo, hi);
      lrow += lo + hi;
    }
    // O^T += V^T P^T over the 16-key groups (keys 16g + ...)
#pragma unroll
    for (int g = 0; g < 2 * NS; ++g) {
      const int t = g >> 1, half = g & 1;   // score tile, and which 16 keys of it
      bf16x8_t pb;
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[j] = (__bf16)sc[t][8 * half + j];
      // keys 16g + 4h + {0..3, 8..11} sit at V^T columns 16g + 8h .. +7
#pragma unroll
      for (int ot = 0; ot < NOT; ++ot) {
        const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(&V_[(ot * 32 + c32) * LDV + 16 * g + 8 * h]);
        o[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb, o[ot], 0, 0, 0);
      }
    }
    // the other buffer held tile kt-1, which every wave finished before the last barrier
    if (kt + 1 < nt) {
      stage(buf ^ 1);
      if (kt + 2 < nt) fetch(kv0 + 2 * KTL);
    }
    FF_LDS_BARRIER();
  }
#undef FF_LDS_BARRIER
  if (SPLIT > 1) {
    // merge the groups' (m, l, O) through LDS (the tile buffers are free after the last
    // barrier): group g > 0 writes, group 0 combines in group order, exactly:
    // m = max m_g, O = sum_g O_g 2^(m_g - m), l = sum_g l_g 2^(m_g - m)
    constexpr int PF = NOT * 16 + 2;   // floats per lane
    float* xch = reinterpret_cast<float*>(smem);
    static_assert(sizeof(smem) >= (size_t)(SPLIT - 1) * NW * 64 * PF * 4, "exchange space");
    if (grp > 0) {
      float* p = xch + (((size_t)(grp - 1) * NW + wave) * PF) * 64 + lane;
#pragma unroll
      for (int t = 0; t < NOT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) p[(t * 16 + v) * 64] = o[t][v];
      p[(NOT * 16) * 64] = mrow;
      p[(NOT * 16 + 1) * 64] = lrow;
    }
    __syncthreads();
    if (grp > 0) return;
#pragma unroll
    for (int g2 = 1; g2 < SPLIT; ++g2) {
      const float* p = xch + (((size_t)(g2 - 1) * NW + wave) * PF) * 64 + lane;
      const float m2 = p[(NOT * 16) * 64], l2 = p[(NOT * 16 + 1) * 64];
      const float mm = fmaxf(mrow, m2);
      const float a1 = __builtin_amdgcn_exp2f(mrow - mm), a2 = __builtin_amdgcn_exp2f(m2 - mm);
#pragma unroll
      for (int t = 0; t < NOT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[t][v] = o[t][v] * a1 + p[(t * 16 + v) * 64] * a2;
      lrow = lrow * a1 + l2 * a2;
      mrow = mm;
    }
  }
  // o[ot][v] = O[query q0 + c32][e = 32 ot + 8 (v/4) + 4 h + v%4].  In that layout a store
  // instruction writes 8 bytes to each of 32 rows (a memory request per row), so the
  // normalised tile goes through the wave's own LDS region as rows of bf16 and is stored
  // as 16-byte row pieces, consecutive lanes on consecutive pieces.  The region is free:
  // every tile read ended before the last barrier, and with SPLIT > 1 it is this wave's
  // own merge entry, which it has finished reading (LDS ops of a wave complete in order).
  constexpr int LDO = DV + 8;                              // staged row pitch (elements)
  constexpr int PFX = SPLIT > 1 ? (NOT * 16 + 2) * 64 * 2 : 0;   // merge entry (elements)
  constexpr int RW = 32 * LDO > PFX ? 32 * LDO : PFX;
  static_assert(sizeof(smem) >= (size_t)NW * RW * 2, "output staging space");
  uint16_t* stg = smem + wave * RW;
  {
    const float inv = 1.0f / lrow;
#pragma unroll
    for (int ot = 0; ot < NOT; ++ot)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int e = 32 * ot + 8 * g + 4 * h;
        u32x2_t w;
        w[0] = pack_bf16x2(o[ot][4 * g] * inv, o[ot][4 * g + 1] * inv);
        w[1] = pack_bf16x2(o[ot][4 * g + 2] * inv, o[ot][4 * g + 3] * inv);
        *reinterpret_cast<u32x2_t*>(stg + c32 * LDO + e) = w;
      }
  }
  // d % 8 == 0 (host check): d/8 pieces per query row
  uint16_t* out = reinterpret_cast<uint16_t*>(a.out);
  const int ppr = d / 8;
  for (int idx = lane; idx < 32 * ppr; idx += 64) {
    const int row = idx / ppr, pc = idx - row * ppr;
    const int qq = q0 + row;
    if (qq < N)
      *reinterpret_cast<u32x4_t*>(out + (rb + qq) * a.ldo + (size_t)hd * d + pc * 8) =
          *reinterpret_cast<const u32x4_t*>(stg + row * LDO + pc * 8);
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
    // a lane's byte offset within a key tile (at most 132 rows of qkv) must fit 32 bits
    if ((uint64_t)a.ldq * 2 * 132 > 0xffffffffull) return hipErrorInvalidValue;
    // 8 wavefronts (256 queries) per workgroup when that still gives >= 256 workgroups;
    // else 4 wavefronts (128 queries), and when even those are fewer than 2 per CU on
    // average, two groups of 4 over the two halves of the keys
    const bool wide = (long)((a.N + 255) / 256) * a.H * a.B >= 256;
    const bool split = !wide && (long)((a.N + 127) / 128) * a.H * a.B < 512 && a.N > KT;
    const long nwg = (long)((a.N + (wide ? 255 : 127)) / (wide ? 256 : 128)) * a.H * a.B;
    if (nwg > 0x7fffffffL) return hipErrorInvalidValue;
    const dim3 grid((unsigned)nwg);   // one dimension: the kernel maps it to (sample, head, query block)
#define FF_ATTN(DQ, DV)                                                              \
    do {                                                                             \
      if (wide) FF_LAUNCH((k_attn32<DQ, DV, 8, 1, 128>), grid, 512, 0, s, a);        \
      else if (split) FF_LAUNCH((k_attn32<DQ, DV, 4, 2, 64>), grid, 512, 0, s, a);   \
      else FF_LAUNCH((k_attn32<DQ, DV, 4, 1, 64>), grid, 256, 0, s, a);              \
    } while (0)
    if (a.d <= 64) FF_ATTN(64, 64);
    else if (a.d <= 80) FF_ATTN(80, 96);
    else if (a.d <= 96) FF_ATTN(96, 96);
    else FF_ATTN(128, 128);
#undef FF_ATTN
  } else {
    dim3 grid((a.N + 63) / 64, a.H, a.B);
    if (a.d <= 64) FF_LAUNCH(k_attn_f32<64>, grid, 64, 0, s, a);
    else FF_LAUNCH(k_attn_f32<128>, grid, 64, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ff
