// The dense parts of the transformer block around the layer (Section 3.1: each block holds
// an RMSNorm, the BSA layer and a SwiGLU): the channel matrix products on the bf16 matrix
// cores with f32 accumulation, RMSNorm forward/backward, SwiGLU forward/backward, and the
// casts, layout changes and deterministic reductions between them.
#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr float kNormEps = 1e-6f;

// ---- matrix products C[M, N] = sum_k A(m, k) B(n, k) ----
//
// Workgroup tiles of 256 x 256 (eight waves of 64 x 128) or 128 x 128 (four waves of
// 64 x 64) in 16 x 16 accumulator tiles, contraction tiles of 64, two LDS stages filled by
// direct global->LDS loads while the other stage feeds the matrix cores (launch_gemm picks
// the tile from the shape).
//   plain form (trans = false): A [M, K] and B [N, K], contraction index fastest; tiles are
//     staged as 128 rows x 64 (row fragments read with ds_read_b128);
//   transposed form (trans = true): A [K, M] and B [K, N], the contraction runs over their
//     rows (the weight gradients dW = dY^T X over tokens); tiles are staged as 64 rows x 128
//     and read with transposing LDS reads (ds_read_b64_tr_b16).
// Accumulator lane L holds C[m0 + L % 16][n0 + 4 (L / 16) + e], e = 0..3 (the B fragment
// is the first MFMA operand), so each lane stores 4 consecutive columns.

// 16-byte chunk swizzle of a staged tile row: 4 or 8 chunks per row (row-fragment reads
// of 16 consecutive rows on distinct banks) or 16 and more chunks per row (transposing
// reads of 8 consecutive rows, chunk pairs on distinct banks).
template <int COLS>
__device__ __forceinline__ int tile_swz(int x) {
  return COLS == 32 ? ((x >> 2) & 3) : COLS == 64 ? (x & 7) : 2 * (x & 7);
}

// Staging of ROWS x COLS tiles of a logical row-major operand into LDS by the NW waves of
// the workgroup. Each wave instruction fills 1 KB of consecutive LDS; lane L's 16 bytes
// land at bytes [16 L, 16 L + 16) and the lane fetches the chunk the swizzle puts there.
// The element offset of that chunk splits into a per-lane part fixed for the kernel and a
// wave-uniform part per contraction tile (kt_offset; shapes are whole tiles, as the
// launcher checks).
template <int ROWS, int COLS, int NW>
struct TileLoader {
  static constexpr int CPR = COLS / 8;
  static constexpr int NU = ROWS * CPR / (64 * NW);   // wave instructions per wave
  static_assert(NU * 64 * NW == ROWS * CPR, "tile / wave split");
  const bf16_t* p;
  long long lane_off[NU];

  // (r0, c0): the tile origin of the operand block this workgroup owns, as (row, column)
  // of the logical matrix at kt = 0.
  __device__ __forceinline__ void init(const GemmMat& m, long long r0, int c0, int wid, int lane) {
    p = reinterpret_cast<const bf16_t*>(m.p);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int idx = (wid * NU + u) * 64 + lane;
      const int row = idx / CPR;
      const int col = 8 * ((idx % CPR) ^ tile_swz<COLS>(row));
      const long long r = r0 + row;
      const int c = c0 + col;
      if (m.heads == 0) {
        lane_off[u] = r * m.ld + c;
      } else {
        const long long b = r >> m.lgn, t = r & ((1LL << m.lgn) - 1);
        lane_off[u] = ((((b * m.heads + (c >> m.lgd)) << m.lgn) + t) << m.lgd) + (c & ((1 << m.lgd) - 1));
      }
    }
  }
  __device__ __forceinline__ void issue(bf16_t* lds, long long kt_off, int wid) const {
#pragma unroll
    for (int u = 0; u < NU; ++u)
      __builtin_amdgcn_global_load_lds(p + kt_off + lane_off[u], lds + (wid * NU + u) * 512, 16, 0, 0);
  }
};

// Wave-uniform element offset of contraction tile kt (BK wide) of an operand.
// Plain form: columns BK kt; in the heads layout a tile stays inside one head (BK <= d) or
// covers whole heads (d divides BK), n d elements per head. Transposed form: rows BK kt;
// in the heads layout BK divides n, so a tile stays inside one cloud.
template <bool TR, int BK>
__device__ __forceinline__ long long kt_offset(const GemmMat& m, int kt) {
  const long long k0 = (long long)kt * BK;
  if (!TR) {
    if (m.heads == 0) return k0;
    return ((k0 >> m.lgd) << (m.lgn + m.lgd)) + (k0 & ((1LL << m.lgd) - 1));
  }
  if (m.heads == 0) return k0 * m.ld;
  const long long b = k0 >> m.lgn, t = k0 & ((1LL << m.lgn) - 1);
  return ((b * m.heads << m.lgn) + t) << m.lgd;
}

template <int BK>
__device__ __forceinline__ bf16x8 frag_row(const bf16_t* t, int row, int lc) {
  return *reinterpret_cast<const bf16x8*>(t + row * BK + 8 * (lc ^ tile_swz<BK>(row)));
}

// Workgroup barrier without a memory fence: the waves' direct-to-LDS loads are already
// waited for by each wave (vmcnt), and later tiles stay in flight across it (the fence of
// __syncthreads would wait for every outstanding load). The empty statements keep the
// compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with vmcnt = V (expcnt and lgkmcnt left at their maxima)
template <int V>
__device__ __forceinline__ void vm_wait() {
  static_assert(V >= 0 && V < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4) | (15 << 8));
}

// LDS byte addresses of the two transposing reads that give lane (p = L % 16, j = L / 16)
// the operand X[k0 + 4j + i][m0 + p] (i = 0..3) and X[k0 + 16 + 4j + i][m0 + p] of a
// [64][COLS] tile X: within each 16-lane group, ds_read_b64_tr_b16 hands lane l element
// l % 4 of the 4-element runs addressed by lanes l / 4, 4 + l / 4, 8 + l / 4, 12 + l / 4, so
// lane p addresses row k0 + 4j + p / 4 (then + 16) at columns m0 + 4 (p % 4) + [0, 4).
template <int COLS>
__device__ __forceinline__ void tr_addr(const bf16_t* t, int k0, int m0, int lane, uint32_t& o0, uint32_t& o1) {
  const int p = lane & 15, j = lane >> 4;
  const int col = m0 + 4 * (p & 3);
  const int lc = col >> 3, sub = col & 7;
  const int x0 = k0 + 4 * j + (p >> 2), x1 = x0 + 16;
  const bf16_t* a0 = t + x0 * COLS + 8 * (lc ^ tile_swz<COLS>(x0)) + sub;
  const bf16_t* a1 = t + x1 * COLS + 8 * (lc ^ tile_swz<COLS>(x1)) + sub;
  o0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)a0;
  o1 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)a1;
}

// Four operand fragments (columns m0 + 16 i, i = 0..3) of one 32-deep contraction step of
// the transposed form, issued as one statement that also waits for them: every use of the
// results follows the wait.
template <int COLS>
__device__ __forceinline__ void tr_frags4(const bf16_t* t, int k0, int m0, int lane, bf16x8 (&f)[4]) {
  uint32_t a[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) tr_addr<COLS>(t, k0, m0 + 16 * i, lane, a[2 * i], a[2 * i + 1]);
  uint2 r[8];
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8\n\tds_read_b64_tr_b16 %1, %9\n\t"
      "ds_read_b64_tr_b16 %2, %10\n\tds_read_b64_tr_b16 %3, %11\n\t"
      "ds_read_b64_tr_b16 %4, %12\n\tds_read_b64_tr_b16 %5, %13\n\t"
      "ds_read_b64_tr_b16 %6, %14\n\tds_read_b64_tr_b16 %7, %15\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
      : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]), "v"(a[7])
      : "memory");
#pragma unroll
  for (int i = 0; i < 4; ++i)
    f[i] = __builtin_bit_cast(bf16x8, make_uint4(r[2 * i].x, r[2 * i].y, r[2 * i + 1].x, r[2 * i + 1].y));
}

struct GemmArgs {
  GemmMat a, b;
  int ntn;        // column tiles
  int kt_per;     // contraction tiles per split
  GemmOut o;
  long long split_stride;   // elements between the partial products of two splits
};

// Workgroup tile BM x BN of WM x WN waves (wave tile BM / WM x BN / WN in 16 x 16
// accumulator tiles); contraction tiles of BK in a ring of NS LDS stages, NS - 1 of them in
// flight while one feeds the matrix cores.
template <bool TR, int BM, int BN, int WM, int WN, int BK, int NS>
__global__ void __launch_bounds__(64 * WM * WN) gemm_kernel(GemmArgs g) {
  constexpr int NW = WM * WN;
  constexpr int TMW = BM / WM, TNW = BN / WN;
  constexpr int FI = TMW / 16, FJ = TNW / 16;
  static_assert(FI % 4 == 0 && FJ % 4 == 0, "wave tile");
  static_assert(NS >= 2 && NS <= 4 && (BK == 32 || BK == 64), "pipeline");
  constexpr int AE = BM * BK, BE = BN * BK;
  __shared__ __attribute__((aligned(1024))) bf16_t as0[AE], bs0[BE], as1[AE], bs1[BE];
  __shared__ __attribute__((aligned(1024))) bf16_t as2[NS > 2 ? AE : 8], bs2[NS > 2 ? BE : 8];
  __shared__ __attribute__((aligned(1024))) bf16_t as3[NS > 3 ? AE : 8], bs3[NS > 3 ? BE : 8];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wm = wid / WN, wn = wid % WN;
  // workgroups are dealt to the 8 XCDs round-robin; give each XCD a contiguous run of
  // tiles (row panels walked column tile by column tile) so it re-reads A from its own L2
  const int nt = gridDim.x;
  int id = blockIdx.x;
  if ((nt & 7) == 0) id = (id & 7) * (nt >> 3) + (id >> 3);
  const int tm = id / g.ntn, tn = id - tm * g.ntn;
  const long long m0 = (long long)tm * BM, n0 = (long long)tn * BN;
  const int kt0 = blockIdx.y * g.kt_per, kt1 = kt0 + g.kt_per;

  TileLoader<TR ? BK : BM, TR ? BM : BK, NW> la;
  TileLoader<TR ? BK : BN, TR ? BN : BK, NW> lb;
  if (!TR) {
    la.init(g.a, m0, 0, wid, lane);
    lb.init(g.b, n0, 0, wid, lane);
  } else {
    la.init(g.a, 0, (int)m0, wid, lane);
    lb.init(g.b, 0, (int)n0, wid, lane);
  }
  constexpr int PER = decltype(la)::NU + decltype(lb)::NU;   // wave load instructions per tile
  bf16_t* const AS[4] = {as0, as1, as2, as3};
  bf16_t* const BS[4] = {bs0, bs1, bs2, bs3};
  auto issue = [&](int kt, int st) {
    la.issue(AS[st], kt_offset<TR, BK>(g.a, kt), wid);
    lb.issue(BS[st], kt_offset<TR, BK>(g.b, kt), wid);
  };
  f32x4 acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const bf16_t* as, const bf16_t* bs) {
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 af[FI], bfr[FJ];
      if (!TR) {
#pragma unroll
        for (int i = 0; i < FI; ++i) af[i] = frag_row<BK>(as, wm * TMW + 16 * i + (lane & 15), 4 * ks + (lane >> 4));
#pragma unroll
        for (int j = 0; j < FJ; ++j) bfr[j] = frag_row<BK>(bs, wn * TNW + 16 * j + (lane & 15), 4 * ks + (lane >> 4));
      } else {
#pragma unroll
        for (int i = 0; i < FI; i += 4)
          tr_frags4<BM>(as, 32 * ks, wm * TMW + 16 * i, lane, *reinterpret_cast<bf16x8(*)[4]>(&af[i]));
#pragma unroll
        for (int j = 0; j < FJ; j += 4)
          tr_frags4<BN>(bs, 32 * ks, wn * TNW + 16 * j, lane, *reinterpret_cast<bf16x8(*)[4]>(&bfr[j]));
      }
#pragma unroll
      for (int i = 0; i < FI; ++i)
#pragma unroll
        for (int j = 0; j < FJ; ++j) acc[i][j] = mma(bfr[j], af[i], acc[i][j]);
    }
  };

#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (kt0 + s < kt1) issue(kt0 + s, s);
  for (int kt = kt0; kt < kt1; kt += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int t = kt + s;
      if (t < kt1) {
        // tile t has landed once at most the NS - 2 tiles issued after it are in flight
        if (t + NS - 2 < kt1)
          vm_wait<(NS - 2) * PER>();
        else
          vm_drain();
        lds_barrier();     // every wave's loads of tile t are visible; stage s - 1 is free
        if (t + NS - 1 < kt1) issue(t + NS - 1, (s + NS - 1) % NS);
        compute(AS[s], BS[s]);
      }
    }
  }

  const GemmOut& o = g.o;
  const int r = lane & 15, jq = lane >> 4;
  auto pack4 = [](float a0, float a1, float a2, float a3) {
    return make_uint2((uint32_t)f2bf(a0) | ((uint32_t)f2bf(a1) << 16), (uint32_t)f2bf(a2) | ((uint32_t)f2bf(a3) << 16));
  };
  if (o.epi == kEpiSwigluFwd) {
    // B rows interleaved in groups of TNW (TNW / 2 rows of W_1, then the same rows of
    // W_3; launch_cast_w13 with gemm_wave_cols): the wave's column tiles j and j + FJ / 2
    // hold u and w of the same hidden units f
    const int F = o.ffn;
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      const long long m = m0 + wm * TMW + 16 * i + r;
#pragma unroll
      for (int j = 0; j < FJ / 2; ++j) {
        const int f = ((int)n0 + wn * TNW) / 2 + 16 * j + 4 * jq;
        float u[4], w[4], a[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          u[e] = bf2f(f2bf(acc[i][j][e]));
          w[e] = bf2f(f2bf(acc[i][j + FJ / 2][e]));
          a[e] = u[e] / (1.0f + __expf(-u[e])) * w[e];
        }
        bf16_t* uw = reinterpret_cast<bf16_t*>(o.out) + m * 2 * F + f;
        *reinterpret_cast<uint2*>(uw) = pack4(u[0], u[1], u[2], u[3]);
        *reinterpret_cast<uint2*>(uw + F) = pack4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<uint2*>(reinterpret_cast<bf16_t*>(o.out2) + m * F + f) = pack4(a[0], a[1], a[2], a[3]);
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < FI; ++i) {
    const long long m = m0 + wm * TMW + 16 * i + r;
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int n = (int)n0 + wn * TNW + 16 * j + 4 * jq;
      f32x4 v = acc[i][j];
      if (o.epi == kEpiF32 || o.epi == kEpiPart) {
        float* dst = reinterpret_cast<float*>(o.out) + (o.epi == kEpiPart ? blockIdx.y * g.split_stride : 0) +
                     m * o.ldc + n;
        if (o.epi == kEpiF32 && o.res) {
          const float4 rv = *reinterpret_cast<const float4*>(o.res + m * o.ldr + n);
          v[0] += rv.x;
          v[1] += rv.y;
          v[2] += rv.z;
          v[3] += rv.w;
        }
        *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
      } else if (o.epi == kEpiSwigluBwd) {
        // v = da for hidden units n .. n + 3; u, w from the forward pass (bf16 [M, 2F])
        const int F = o.ffn;
        const bf16_t* uwp = reinterpret_cast<const bf16_t*>(o.aux) + m * 2 * F + n;
        const uint2 ub = *reinterpret_cast<const uint2*>(uwp), wb = *reinterpret_cast<const uint2*>(uwp + F);
        const uint32_t uu[2] = {ub.x, ub.y}, ww[2] = {wb.x, wb.y};
        float du[4], dw[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float uf = __uint_as_float((uu[e >> 1] >> (16 * (e & 1))) << 16);
          const float wf = __uint_as_float((ww[e >> 1] >> (16 * (e & 1))) << 16);
          const float sg = 1.0f / (1.0f + __expf(-uf));
          du[e] = v[e] * wf * sg * (1.0f + uf * (1.0f - sg));
          dw[e] = v[e] * uf * sg;
        }
        bf16_t* dst = reinterpret_cast<bf16_t*>(o.out) + m * 2 * F + n;
        *reinterpret_cast<uint2*>(dst) = pack4(du[0], du[1], du[2], du[3]);
        *reinterpret_cast<uint2*>(dst + F) = pack4(dw[0], dw[1], dw[2], dw[3]);
      } else {
        bf16_t* dst;
        if (o.epi == kEpiBf16) {
          dst = reinterpret_cast<bf16_t*>(o.out) + m * o.ldc + n;
        } else {   // kEpiHeads
          const int p = n / o.part_cols, c = n - p * o.part_cols;
          const long long b = m >> o.lgn, t = m & ((1LL << o.lgn) - 1);
          const long long h = c >> o.lgd, dd = c & ((1 << o.lgd) - 1);
          dst = reinterpret_cast<bf16_t*>(o.parts[p]) + ((((b * o.heads + h) << o.lgn) + t) << o.lgd) + dd;
        }
        *reinterpret_cast<uint2*>(dst) = pack4(v[0], v[1], v[2], v[3]);
      }
    }
  }
}

// ---- RMSNorm: one wave per row; lane L holds columns 2L + 128 t, t < C / 128 ----

template <int CT>
__global__ void __launch_bounds__(256) rmsnorm_fwd_kernel(const float* __restrict__ x, const float* __restrict__ gain,
                                                          const float* __restrict__ wg, long long rows,
                                                          bf16_t* __restrict__ xn, float* __restrict__ rstd,
                                                          float* __restrict__ gate) {
  constexpr int C = 128 * CT;
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float* xr = x + row * C;
  float2 v[CT];
  float ss = 0.f;
#pragma unroll
  for (int t = 0; t < CT; ++t) {
    v[t] = *reinterpret_cast<const float2*>(xr + 128 * t + 2 * lane);
    ss += v[t].x * v[t].x + v[t].y * v[t].y;
  }
  ss = wave_sum(ss);
  const float rs = 1.0f / sqrtf(ss / (float)C + kNormEps);
  float gd[3] = {0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < CT; ++t) {
    const int c = 128 * t + 2 * lane;
    const float2 gg = *reinterpret_cast<const float2*>(gain + c);
    const float a0 = v[t].x * rs * gg.x, a1 = v[t].y * rs * gg.y;
    *reinterpret_cast<uint32_t*>(xn + row * C + c) = (uint32_t)f2bf(a0) | ((uint32_t)f2bf(a1) << 16);
    if (wg) {
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) {
        const float2 w = *reinterpret_cast<const float2*>(wg + jj * C + c);
        gd[jj] += a0 * w.x + a1 * w.y;
      }
    }
  }
  if (wg) {
#pragma unroll
    for (int jj = 0; jj < 3; ++jj) gd[jj] = wave_sum(gd[jj]);
    if (lane == 0) {
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) gate[row * 3 + jj] = gd[jj];
    }
  }
  if (lane == 0) rstd[row] = rs;
}

// dx = dres + r (dxh - xh mean(dxh xh)) with xh = x r, dxh = (dxn + dgate W_g) g, per row.
// Workgroup b owns a contiguous run of rows (wave w takes every fourth row from w); the
// sums over its rows of dg = (dxn + dgate W_g) xh and dW_g = dgate (xh g) go to
// part[b][4C] (dg, then dW_g row by row; zero without dgate), the four waves' sums added in
// wave order.
template <int CT>
__global__ void __launch_bounds__(256) rmsnorm_bwd_kernel(const float* __restrict__ dxn, const float* __restrict__ x,
                                                          const float* __restrict__ rstd, const float* __restrict__ gain,
                                                          const float* __restrict__ dres, const float* __restrict__ dgate,
                                                          const float* __restrict__ wg, long long rows, int rpg,
                                                          float* __restrict__ dx, bf16_t* __restrict__ dx16,
                                                          float* __restrict__ part) {
  constexpr int C = 128 * CT;
  __shared__ float red[3][4 * C];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const long long g0 = (long long)blockIdx.x * rpg, g1 = g0 + rpg < rows ? g0 + rpg : rows;
  float2 gg[CT], ag[CT], w[3][CT], aw[3][CT];
#pragma unroll
  for (int t = 0; t < CT; ++t) {
    const int c = 128 * t + 2 * lane;
    gg[t] = *reinterpret_cast<const float2*>(gain + c);
    ag[t] = make_float2(0.f, 0.f);
#pragma unroll
    for (int jj = 0; jj < 3; ++jj) {
      w[jj][t] = dgate ? *reinterpret_cast<const float2*>(wg + jj * C + c) : make_float2(0.f, 0.f);
      aw[jj][t] = make_float2(0.f, 0.f);
    }
  }
  for (long long row = g0 + wid; row < g1; row += 4) {
    const float rs = rstd[row];
    float dga[3] = {0.f, 0.f, 0.f};
    if (dgate) {
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) dga[jj] = dgate[row * 3 + jj];
    }
    float2 dn[CT], xh[CT], dr[CT];
    float s = 0.f;
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = 128 * t + 2 * lane;
      dn[t] = *reinterpret_cast<const float2*>(dxn + row * C + c);
      dr[t] = *reinterpret_cast<const float2*>(dres + row * C + c);
      const float2 xv = *reinterpret_cast<const float2*>(x + row * C + c);
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) {
        dn[t].x += dga[jj] * w[jj][t].x;
        dn[t].y += dga[jj] * w[jj][t].y;
      }
      xh[t] = make_float2(xv.x * rs, xv.y * rs);
      s += dn[t].x * gg[t].x * xh[t].x + dn[t].y * gg[t].y * xh[t].y;
      ag[t].x += dn[t].x * xh[t].x;
      ag[t].y += dn[t].y * xh[t].y;
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) {
        aw[jj][t].x += dga[jj] * xh[t].x * gg[t].x;
        aw[jj][t].y += dga[jj] * xh[t].y * gg[t].y;
      }
    }
    s = wave_sum(s) / (float)C;
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = 128 * t + 2 * lane;
      const float d0 = rs * (dn[t].x * gg[t].x - xh[t].x * s) + dr[t].x;
      const float d1 = rs * (dn[t].y * gg[t].y - xh[t].y * s) + dr[t].y;
      *reinterpret_cast<float2*>(dx + row * C + c) = make_float2(d0, d1);
      if (dx16) *reinterpret_cast<uint32_t*>(dx16 + row * C + c) = (uint32_t)f2bf(d0) | ((uint32_t)f2bf(d1) << 16);
    }
  }
  if (wid > 0) {
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = 128 * t + 2 * lane;
      *reinterpret_cast<float2*>(&red[wid - 1][c]) = ag[t];
#pragma unroll
      for (int jj = 0; jj < 3; ++jj) *reinterpret_cast<float2*>(&red[wid - 1][(1 + jj) * C + c]) = aw[jj][t];
    }
  }
  __syncthreads();
  if (wid == 0) {
    float* pw = part + (long long)blockIdx.x * 4 * C;
#pragma unroll
    for (int t = 0; t < CT; ++t) {
      const int c = 128 * t + 2 * lane;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float2 v = q == 0 ? ag[t] : aw[q - 1][t];
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          const float2 o = *reinterpret_cast<const float2*>(&red[k][q * C + c]);
          v.x += o.x;
          v.y += o.y;
        }
        *reinterpret_cast<float2*>(pw + q * C + c) = v;
      }
    }
  }
}

// out[by * ncols + c] = sum over rows p in [32 by, 32 by + 32) (below P) of
// part[p * ld + col0 + c], c < ncols; wave w sums rows 32 by + 8 w .. + 8 and the four
// waves' sums are added in wave order.
__global__ void __launch_bounds__(256) colsum_kernel(const float* __restrict__ part, int P, long long ld, int col0,
                                                     int ncols, float* __restrict__ out) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + lane;
  const int p0 = blockIdx.y * 32 + w * 8;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = c < ncols && p0 + i < P ? part[(long long)(p0 + i) * ld + col0 + c] : 0.f;
  float s = v[0];
#pragma unroll
  for (int i = 1; i < 8; ++i) s += v[i];
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && c < ncols) out[(long long)blockIdx.y * ncols + c] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

// out[i] = sum over s of part[s * stride + i], four elements per thread, splits in order.
__global__ void __launch_bounds__(256) splitk_sum_kernel(const float* __restrict__ part, int S, long long stride,
                                                         long long count4, float* __restrict__ out) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= count4) return;
  float4 s = reinterpret_cast<const float4*>(part)[i];
  for (int k = 1; k < S; ++k) {
    const float4 v = reinterpret_cast<const float4*>(part + k * stride)[i];
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
  }
  reinterpret_cast<float4*>(out)[i] = s;
}

// [M, 3C] bf16 token-major rows from dq, dk, dv [B, H, N, d] f32, eight elements per thread.
__global__ void __launch_bounds__(256) pack_qkv_kernel(const float* __restrict__ dq, const float* __restrict__ dk,
                                                       const float* __restrict__ dv, long long rows, int C, int H,
                                                       int lgn, int lgd, bf16_t* __restrict__ out) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const int c8 = 3 * C / 8;
  if (idx >= rows * c8) return;
  const long long m = idx / c8;
  const int col = (int)(idx - m * c8) * 8;
  const int p = col / C, c = col - p * C;
  const float* src = p == 0 ? dq : (p == 1 ? dk : dv);
  const long long b = m >> lgn, t = m & ((1LL << lgn) - 1);
  const long long h = c >> lgd, dd = c & ((1 << lgd) - 1);
  const f32x8 v = load_chunk(src + ((((b * H + h) << lgn) + t) << lgd) + dd);
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = v[e];
  *reinterpret_cast<bf16x8*>(out + m * 3 * C + col) = make_chunk<bf16_t>(o);
}

__global__ void __launch_bounds__(256) cast_bf16_kernel(const float* __restrict__ src, long long n8,
                                                        bf16_t* __restrict__ dst) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const f32x8 v = load_chunk(src + 8 * i);
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = v[e];
  *reinterpret_cast<bf16x8*>(dst + 8 * i) = make_chunk<bf16_t>(o);
}

// dst[c * ldd + r] = bf16(src[r * cols + c]) for a [rows, cols] f32 matrix (32 x 32 tiles
// through LDS; rows and cols multiples of 32).
__global__ void __launch_bounds__(256) cast_t_kernel(const float* __restrict__ src, int rows, int cols,
                                                     bf16_t* __restrict__ dst, long long ldd) {
  __shared__ float tile[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
#pragma unroll
  for (int k = 0; k < 4; ++k) tile[ty + 8 * k][tx] = src[(long long)(r0 + ty + 8 * k) * cols + c0 + tx];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 4; ++k) dst[(long long)(c0 + ty + 8 * k) * ldd + r0 + tx] = f2bf(tile[tx][ty + 8 * k]);
}

// dst rows of the interleaved [W_1; W_3] operand in groups of G rows: row r takes row
// (G / 2)(r / G) + r % G of W_1 when r % G < G / 2, else row (G / 2)(r / G) + r % G - G / 2
// of W_3 (f32 -> bf16, eight elements per thread; C a multiple of 8).
__global__ void __launch_bounds__(256) cast_w13_kernel(const float* __restrict__ w1, const float* __restrict__ w3,
                                                       int F, int C, int G, bf16_t* __restrict__ dst) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  const int c8 = C / 8;
  if (i >= 2LL * F * c8) return;
  const long long r = i / c8;
  const int c = (int)(i - r * c8) * 8;
  const int g = (int)(r / G), wi = (int)(r % G), h = G / 2;
  const float* src = wi < h ? w1 + (long long)(h * g + wi) * C : w3 + (long long)(h * g + wi - h) * C;
  const f32x8 v = load_chunk(src + c);
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = v[e];
  *reinterpret_cast<bf16x8*>(dst + r * C + c) = make_chunk<bf16_t>(o);
}

unsigned blocks_for(long long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

// 256 x 256 workgroup tiles of 8 waves (4 x 2, 64 x 128 each) where the shape allows and
// gives at least 256 tiles (or splits the contraction), else 128 x 128 tiles of 4 waves
// (64 x 64 each); contraction tiles of 64 in two stages. (Measured on the block's shapes:
// 256 x 256 tiles of 4 x 2 waves ran fastest, ahead of 2 x 4 waves, 256 x 128 and
// 128 x 256 tiles, and of 32-deep tiles in four stages.)
int gemm_tile(int M, int N, bool split) {
  return M % 256 == 0 && N % 256 == 0 && (split || (long long)(M / 256) * (N / 256) >= 256) ? 256 : 128;
}

hipError_t launch_gemm(bool trans, const GemmMat& a, const GemmMat& b, int M, int N, long long K, int splits,
                       const GemmOut& o, hipStream_t st) {
  if (M <= 0 || N <= 0 || K <= 0 || M % 128 || N % 128 || K % 64 || splits < 1 || (K / 64) % splits)
    return hipErrorInvalidValue;
  if (o.epi != kEpiPart && splits != 1) return hipErrorInvalidValue;
  const int T = gemm_tile(M, N, trans);
  GemmArgs g{a, b, N / T, (int)((K / 64) / splits), o, (long long)M * o.ldc};
  const dim3 grid((unsigned)((M / T) * (N / T)), (unsigned)splits);
  if (T == 256) {
    if (trans)
      gemm_kernel<true, 256, 256, 4, 2, 64, 2><<<grid, 512, 0, st>>>(g);
    else
      gemm_kernel<false, 256, 256, 4, 2, 64, 2><<<grid, 512, 0, st>>>(g);
  } else {
    if (trans)
      gemm_kernel<true, 128, 128, 2, 2, 64, 2><<<grid, 256, 0, st>>>(g);
    else
      gemm_kernel<false, 128, 128, 2, 2, 64, 2><<<grid, 256, 0, st>>>(g);
  }
  return hipGetLastError();
}

int gemm_wave_cols(int M, int N) { return gemm_tile(M, N, false) == 256 ? 128 : 64; }

int gemm_splits(int M, int N, long long K) {
  const int T = gemm_tile(M, N, true);
  const long long tiles = (long long)(M / T) * (N / T);
  const long long nkt = K / 64;
  int s = 1;
  // about one workgroup per CU (each split adds a partial product the sum reads back), at
  // least 16 contraction tiles per split
  while (tiles * s < 256 && nkt % (2 * s) == 0 && nkt / (2 * s) >= 16) s *= 2;
  return s;
}

hipError_t launch_rmsnorm_fwd(const float* x, const float* gain, const float* wg, long long rows, int C, uint16_t* xn,
                              float* rstd, float* gate, hipStream_t st) {
  const unsigned nb = blocks_for(rows, 4);
  bf16_t* o = reinterpret_cast<bf16_t*>(xn);
  switch (C) {
    case 128: rmsnorm_fwd_kernel<1><<<nb, 256, 0, st>>>(x, gain, wg, rows, o, rstd, gate); break;
    case 256: rmsnorm_fwd_kernel<2><<<nb, 256, 0, st>>>(x, gain, wg, rows, o, rstd, gate); break;
    case 512: rmsnorm_fwd_kernel<4><<<nb, 256, 0, st>>>(x, gain, wg, rows, o, rstd, gate); break;
    case 1024: rmsnorm_fwd_kernel<8><<<nb, 256, 0, st>>>(x, gain, wg, rows, o, rstd, gate); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// row groups of the RMSNorm backward: up to 1024 workgroups, at least 16 rows each
int rmsnorm_bwd_groups(long long rows) {
  const long long g = (rows + 15) / 16;
  return (int)(g < 1024 ? g : 1024);
}

// deterministic column sums of part [P][ld] (columns col0 .. col0 + ncols - 1) into out, in
// two levels (32-row partial sums in tmp [ceil(P / 32)][ncols], then their sum)
hipError_t colsum(const float* part, int P, long long ld, int col0, int ncols, float* tmp, float* out, hipStream_t st) {
  const int rs = (P + 31) / 32;
  if (rs == 1) {
    colsum_kernel<<<dim3(blocks_for(ncols, 64), 1), 256, 0, st>>>(part, P, ld, col0, ncols, out);
    return hipGetLastError();
  }
  colsum_kernel<<<dim3(blocks_for(ncols, 64), rs), 256, 0, st>>>(part, P, ld, col0, ncols, tmp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return colsum(tmp, rs, ncols, 0, ncols, tmp + (long long)rs * ncols, out, st);
}

hipError_t launch_rmsnorm_bwd(const float* dxn, const float* x, const float* rstd, const float* gain, const float* dres,
                              const float* dgate, const float* wg, long long rows, int C, float* dx, uint16_t* dx16,
                              float* part, float* dgain, float* dwg, hipStream_t st) {
  const int ng = rmsnorm_bwd_groups(rows);
  const int rpg = (int)((rows + ng - 1) / ng);
  bf16_t* o16 = reinterpret_cast<bf16_t*>(dx16);
  switch (C) {
    case 128: rmsnorm_bwd_kernel<1><<<ng, 256, 0, st>>>(dxn, x, rstd, gain, dres, dgate, wg, rows, rpg, dx, o16, part); break;
    case 256: rmsnorm_bwd_kernel<2><<<ng, 256, 0, st>>>(dxn, x, rstd, gain, dres, dgate, wg, rows, rpg, dx, o16, part); break;
    case 512: rmsnorm_bwd_kernel<4><<<ng, 256, 0, st>>>(dxn, x, rstd, gain, dres, dgate, wg, rows, rpg, dx, o16, part); break;
    case 1024: rmsnorm_bwd_kernel<8><<<ng, 256, 0, st>>>(dxn, x, rstd, gain, dres, dgate, wg, rows, rpg, dx, o16, part); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  float* tmp = part + (long long)ng * 4 * C;
  e = colsum(part, ng, 4LL * C, 0, C, tmp, dgain, st);
  if (e != hipSuccess || !dgate) return e;
  return colsum(part, ng, 4LL * C, C, 3 * C, tmp, dwg, st);
}

size_t rmsnorm_bwd_part_bytes(long long rows, int C) {
  // partial rows, then the first level of the column sums (at most 32 rows) and the second
  const long long ng = rmsnorm_bwd_groups(rows);
  return sizeof(float) * (size_t)(ng + 32 + 1) * 4 * C;
}

hipError_t launch_splitk_sum(const float* part, int S, long long stride, long long count, float* out, hipStream_t st) {
  if (count % 4 || stride % 4) return hipErrorInvalidValue;
  splitk_sum_kernel<<<blocks_for(count / 4, 256), 256, 0, st>>>(part, S, stride, count / 4, out);
  return hipGetLastError();
}

hipError_t launch_pack_qkv(const float* dq, const float* dk, const float* dv, long long rows, int C, int H, int lgn,
                           int lgd, uint16_t* out, hipStream_t st) {
  if (C % 8) return hipErrorInvalidValue;
  pack_qkv_kernel<<<blocks_for(rows * (3 * C / 8), 256), 256, 0, st>>>(dq, dk, dv, rows, C, H, lgn, lgd,
                                                                        reinterpret_cast<bf16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_cast_bf16(const float* src, long long n, uint16_t* dst, hipStream_t st) {
  if (n % 8) return hipErrorInvalidValue;
  cast_bf16_kernel<<<blocks_for(n / 8, 256), 256, 0, st>>>(src, n / 8, reinterpret_cast<bf16_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_cast_w13(const float* w1, const float* w3, int F, int C, int G, uint16_t* dst, hipStream_t st) {
  if (G <= 0 || G % 2 || (2 * F) % G || C % 8) return hipErrorInvalidValue;
  cast_w13_kernel<<<blocks_for(2LL * F * (C / 8), 256), 256, 0, st>>>(w1, w3, F, C, G, reinterpret_cast<bf16_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_cast_t(const float* src, int rows, int cols, uint16_t* dst, long long ldd, hipStream_t st) {
  if (rows % 32 || cols % 32) return hipErrorInvalidValue;
  cast_t_kernel<<<dim3(cols / 32, rows / 32), 256, 0, st>>>(src, rows, cols, reinterpret_cast<bf16_t*>(dst), ldd);
  return hipGetLastError();
}

}  // namespace bsa
