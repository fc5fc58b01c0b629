// Building blocks shared by the forward and backward attention kernels: packed
// LDS/global moves, V^T-style transposed staging, and the wave-level online-softmax
// step of the forward pass (see attn_fwd.hip for the formulation).
#pragma once
#include "common.hpp"

namespace bsa {
namespace {

constexpr int kKT = 64;       // keys per LDS tile of the dense kernels
constexpr int kMaxSub = 256;  // 16-key sub-blocks per selection wave (G * k* * l' / 16)
constexpr float kNegInf = -__builtin_huge_valf();

// Two runs of 4 consecutive elements (at p and p + 16) as one 8-element chunk.
__device__ __forceinline__ bf16x8 load_4x2(const bf16_t* p) {
  uint2 a = *reinterpret_cast<const uint2*>(p);
  uint2 b = *reinterpret_cast<const uint2*>(p + 16);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}
__device__ __forceinline__ f32x8 load_4x2(const float* p) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 16);
  return f32x8{a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
}
__device__ __forceinline__ void store4(bf16_t* dst, f32x4 v, float sc) {
  uint32_t lo = (uint32_t)f2bf(v[0] * sc) | ((uint32_t)f2bf(v[1] * sc) << 16);
  uint32_t hi = (uint32_t)f2bf(v[2] * sc) | ((uint32_t)f2bf(v[3] * sc) << 16);
  *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
}
__device__ __forceinline__ void store4(float* dst, f32x4 v, float sc) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0] * sc, v[1] * sc, v[2] * sc, v[3] * sc);
}
// Stage 4 rows x 8 columns of V (row pointers may be null = zero rows) into V^T: one
// 16-byte (bf16) or two 16-byte (f32) loads per row, then 8 packed 4-key column writes.
__device__ __forceinline__ void stage_vt(const bf16_t* const (&rows)[4], int dc, bf16_t* vt, int vstr, int key_off) {
  uint32_t w[4][4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    uint4 t = rows[u] ? *reinterpret_cast<const uint4*>(rows[u] + dc) : make_uint4(0, 0, 0, 0);
    w[u][0] = t.x; w[u][1] = t.y; w[u][2] = t.z; w[u][3] = t.w;
  }
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int wd = x >> 1;
    uint32_t lo, hi;
    if (x & 1) {
      lo = (w[0][wd] >> 16) | (w[1][wd] & 0xFFFF0000u);
      hi = (w[2][wd] >> 16) | (w[3][wd] & 0xFFFF0000u);
    } else {
      lo = (w[0][wd] & 0xFFFFu) | (w[1][wd] << 16);
      hi = (w[2][wd] & 0xFFFFu) | (w[3][wd] << 16);
    }
    *reinterpret_cast<uint2*>(vt + (dc + x) * vstr + key_off) = make_uint2(lo, hi);
  }
}
__device__ __forceinline__ void stage_vt(const float* const (&rows)[4], int dc, float* vt, int vstr, int key_off) {
  float w[4][8];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
    if (rows[u]) {
      a = *reinterpret_cast<const float4*>(rows[u] + dc);
      b = *reinterpret_cast<const float4*>(rows[u] + dc + 4);
    }
    w[u][0] = a.x; w[u][1] = a.y; w[u][2] = a.z; w[u][3] = a.w;
    w[u][4] = b.x; w[u][5] = b.y; w[u][6] = b.z; w[u][7] = b.w;
  }
#pragma unroll
  for (int x = 0; x < 8; ++x)
    *reinterpret_cast<float4*>(vt + (dc + x) * vstr + key_off) = make_float4(w[0][x], w[1][x], w[2][x], w[3][x]);
}

// Same as stage_vt for an explicit base pointer per row (columns [dc, dc+8)).
template <typename T>
__device__ __forceinline__ void stage_t(const T* const (&rows)[4], int dc, T* dst, int stride, int off) {
  stage_vt(rows, dc, dst, stride, off);
}


// ---- register-prefetched staging of a 64-row tile (rows [t0, t0 + 64) of a [*, HD] matrix) ----
// Row-major copy: RV 16-byte vectors per thread. Transposed copy (rows become columns):
// each of the first (64/4)*(HD/4) threads moves a 4-row x 4-column block.
template <typename T> struct Vec4T;
template <> struct Vec4T<bf16_t> { typedef uint2 type; };
template <> struct Vec4T<float> { typedef float4 type; };

template <typename T, int HD, int ROWS = kKT, int NT = 256>
struct TileIO {
  static constexpr int VPR = HD * (int)sizeof(T) / 16;           // 16-byte vectors per row
  static constexpr int RV = (ROWS * VPR + NT - 1) / NT;          // row vectors per thread
  static constexpr int TI = (ROWS / 4) * (HD / 4);               // transposed 4x4 items
  static constexpr int TV = (TI + NT - 1) / NT;                  // transposed items per thread
  typedef typename Vec4T<T>::type V4;

  __device__ static void load_rows(uint4 (&r)[RV], const T* base, int t0, int nrows) {
    if (t0 + ROWS <= nrows) {   // full tile (uniform): no per-load bounds checks
#pragma unroll
      for (int u = 0; u < RV; ++u) {
        const int e = threadIdx.x + NT * u;
        const int row = e / VPR, c = (e % VPR) * (16 / (int)sizeof(T));
        if (ROWS * VPR % NT == 0 || e < ROWS * VPR)
          r[u] = *reinterpret_cast<const uint4*>(base + (size_t)(t0 + row) * HD + c);
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < RV; ++u) {
      const int e = threadIdx.x + NT * u;
      const int row = e / VPR, c = (e % VPR) * (16 / (int)sizeof(T));
      r[u] = make_uint4(0, 0, 0, 0);
      if (e < ROWS * VPR && t0 + row < nrows) r[u] = *reinterpret_cast<const uint4*>(base + (size_t)(t0 + row) * HD + c);
    }
  }
  __device__ static void store_rows(const uint4 (&r)[RV], T* lds, int stride) {
#pragma unroll
    for (int u = 0; u < RV; ++u) {
      const int e = threadIdx.x + NT * u;
      const int row = e / VPR, c = (e % VPR) * (16 / (int)sizeof(T));
      if (e < ROWS * VPR) *reinterpret_cast<uint4*>(lds + row * stride + c) = r[u];
    }
  }
  __device__ static void load_tr(V4 (&r)[TV][4], const T* base, int t0, int nrows) {
    if (t0 + ROWS <= nrows) {   // full tile (uniform): no per-load bounds checks
#pragma unroll
      for (int w = 0; w < TV; ++w) {
        const int it = threadIdx.x + NT * w;
        const int kq = it / (HD / 4), dq = it % (HD / 4);
        if (TI % NT == 0 || it < TI) {
#pragma unroll
          for (int u = 0; u < 4; ++u)
            r[w][u] = *reinterpret_cast<const V4*>(base + (size_t)(t0 + 4 * kq + u) * HD + 4 * dq);
        }
      }
      return;
    }
#pragma unroll
    for (int w = 0; w < TV; ++w) {
      const int it = threadIdx.x + NT * w;
      const int kq = it / (HD / 4), dq = it % (HD / 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int row = t0 + 4 * kq + u;
        r[w][u] = V4{};
        if (it < TI && row < nrows) r[w][u] = *reinterpret_cast<const V4*>(base + (size_t)row * HD + 4 * dq);
      }
    }
  }
  __device__ static void store_tr(const V4 (&r)[TV][4], T* lds, int stride) {
#pragma unroll
    for (int w = 0; w < TV; ++w) {
      const int it = threadIdx.x + NT * w;
      if (it >= TI) continue;
      const int kq = it / (HD / 4), dq = it % (HD / 4);
      store_tr4(r[w], lds + (4 * dq) * stride + 4 * kq, stride);
    }
  }
  // 4x4 transpose: column x of the rows -> 4 consecutive elements of LDS row x
  __device__ static void store_tr4(const uint2 (&r)[4], bf16_t* dst, int stride) {
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int sh = 16 * (x & 1);
      uint32_t e[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) e[u] = ((x < 2 ? r[u].x : r[u].y) >> sh) & 0xFFFFu;
      *reinterpret_cast<uint2*>(dst + x * stride) = make_uint2(e[0] | (e[1] << 16), e[2] | (e[3] << 16));
    }
  }
  __device__ static void store_tr4(const float4 (&r)[4], float* dst, int stride) {
    *reinterpret_cast<float4*>(dst + 0 * stride) = make_float4(r[0].x, r[1].x, r[2].x, r[3].x);
    *reinterpret_cast<float4*>(dst + 1 * stride) = make_float4(r[0].y, r[1].y, r[2].y, r[3].y);
    *reinterpret_cast<float4*>(dst + 2 * stride) = make_float4(r[0].z, r[1].z, r[2].z, r[3].z);
    *reinterpret_cast<float4*>(dst + 3 * stride) = make_float4(r[0].w, r[1].w, r[2].w, r[3].w);
  }
};

// ---- bf16 tiles staged without registers: direct global->LDS loads, transpose reads ----
// A tile of rows x HD bf16 lives in LDS row-major without padding; the 16-byte chunk c of
// row x is stored at chunk c ^ swz(x). The swizzle was chosen by measuring LDS bank
// conflicts on gfx950 (SQ_LDS_BANK_CONFLICT): with it both access patterns below, row
// fragments (ds_read_b128, 16 lanes = 16 consecutive rows) and transpose reads
// (ds_read_b64_tr_b16, 16 lanes = 4 consecutive rows x two chunks), run conflict-free, at
// 4 and 2 cycles per instruction.
// 128-wide rows (f32 rows of 64) are read as row fragments: 16 consecutive rows on
// distinct banks with c ^ (x mod 16). Wider rows are only read by transpose reads; for
// them chunk pairs of 8 consecutive rows land on distinct banks with c ^ 2 (x mod 8).
// Workgroups are dealt to the 8 XCDs round-robin by linear id, and each XCD has its own
// L2. When runs of `per` consecutive x-tiles (within one y, z) read the same rows (the
// query tiles of one ball; every key tile of one query chunk; every query tile of one
// head's compressed keys), the grid is renumbered so that each XCD takes whole runs, in
// order: the shared rows then enter that XCD's L2 once instead of once per XCD. The
// renumbering is a bijection of the grid; it needs gridDim.x % per == 0 and the run count
// to be a multiple of 8, else the grid is kept.
// The same renumbering for a workgroup given by its linear id in a grid of the given
// shape (a grid that is one part of a launch; its first workgroup's id is a multiple of 8).
__device__ __forceinline__ dim3 xcd_grouped_block_at(unsigned lin, dim3 g, int per) {
  constexpr unsigned kXcds = 8;
  const unsigned nx = g.x, ny = g.y;
  const unsigned runs = nx * ny * g.z / (unsigned)max(per, 1);
  if (per <= 1 || nx % (unsigned)per != 0 || runs % kXcds != 0) return dim3(lin % nx, (lin / nx) % ny, lin / (nx * ny));
  const unsigned slot = lin / kXcds;
  const unsigned l = ((lin % kXcds) * (runs / kXcds) + slot / per) * per + slot % per;
  return dim3(l % nx, (l / nx) % ny, l / (nx * ny));
}
__device__ __forceinline__ dim3 xcd_grouped_block(int per) {
  return xcd_grouped_block_at(blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z), gridDim, per);
}

template <int HD>
__device__ __forceinline__ int swz(int x) {
  static_assert(HD == 32 || HD == 64 || HD == 128 || HD >= 256, "tile width");
  return HD == 64 ? (x & 7) : HD == 32 ? ((x >> 1) & 3) : HD == 128 ? (x & 15) : 2 * (x & 7);
}

// Rows [r0, r0 + ROWS) of a row-major [nrows, HD] matrix into an LDS tile, by NW waves.
// Each wave instruction moves 64 lanes x 16 bytes into 1 KB of consecutive LDS (lane L
// fills bytes [16L, 16L + 16)); the lane picks the global chunk that belongs there. Rows
// at or past nrows repeat row nrows - 1 (the caller masks them). Completion is tracked by
// vmcnt: vm_drain() and a barrier make the tile visible to the workgroup.
template <int HD, int ROWS, int NW>
__device__ __forceinline__ void dma_tile(bf16_t* lds, const bf16_t* g, int r0, int nrows, int wid, int lane) {
  constexpr int CPR = HD / 8;           // 16-byte chunks per row
  constexpr int NI = ROWS * CPR / 64;   // 1 KB wave instructions per tile
  static_assert(NI % NW == 0 || NW % NI == 0, "tile / wave split");
  constexpr int PER = NI >= NW ? NI / NW : 1;   // fewer instructions than waves: one each
  if (NI < NW && wid >= NI) return;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int blk = wid * PER + u;
    const int idx = blk * 64 + lane;
    const int row = idx / CPR;
    const int lc = (idx % CPR) ^ swz<HD>(row);
    const int gr = r0 + row < nrows ? r0 + row : nrows - 1;
    __builtin_amdgcn_global_load_lds(g + (size_t)gr * HD + 8 * lc, lds + blk * 512, 16, 0, 0);
  }
}

// dma_tile for a tile known to lie inside the matrix: `g` points at the tile's first row.
// A lane's offset inside the tile depends only on its wave and lane, so the compiler keeps
// it in a register across tiles; per tile only the scalar base moves (no per-row clamp).
template <int HD, int ROWS, int NW>
__device__ __forceinline__ void dma_tile_full(bf16_t* lds, const bf16_t* g, int wid, int lane) {
  constexpr int CPR = HD / 8;
  constexpr int NI = ROWS * CPR / 64;
  static_assert(NI % NW == 0 || NW % NI == 0, "tile / wave split");
  constexpr int PER = NI >= NW ? NI / NW : 1;
  if (NI < NW && wid >= NI) return;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int blk = wid * PER + u;
    const int idx = blk * 64 + lane;
    const int row = idx / CPR;
    const int lc = (idx % CPR) ^ swz<HD>(row);
    __builtin_amdgcn_global_load_lds(g + (row * HD + 8 * lc), lds + blk * 512, 16, 0, 0);
  }
}

// 8 consecutive elements of row x starting at logical chunk lc (an MFMA row fragment).
template <int HD>
__device__ __forceinline__ bf16x8 lds_row_chunk(const bf16_t* t, int x, int lc) {
  return *reinterpret_cast<const bf16x8*>(t + x * HD + 8 * (lc ^ swz<HD>(x)));
}

// MFMA A operand of the transposed tile, in the contraction order of a probability chunk
// built from two 16-key accumulator tiles (elements 0-3: keys 4j + i of the first tile,
// 4-7: keys 4j + i of the second): lane (r = lane % 16, j = lane / 16) receives
// X[k0 + 4j + i][m0 + r] and X[k0 + 16 + 4j + i][m0 + r], i = 0..3, from the row-major
// tile X, with two ds_read_b64_tr_b16. Within each 16-lane group that
// instruction hands lane l element l % 4 of the 4-element runs addressed by lanes l / 4,
// 4 + l / 4, 8 + l / 4, 12 + l / 4; lane p therefore addresses row k0 + 4j + p / 4 (then
// + 16), columns m0 + 4 (p % 4) + [0, 4).
template <int HD>
__device__ __forceinline__ bf16x8 lds_tr_chunk(const bf16_t* t, int k0, int m0, int lane) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const int p = lane & 15, j = lane >> 4;
  const int col = m0 + 4 * (p & 3);
  const int lc = col >> 3, sub = col & 7;
  const int x0 = k0 + 4 * j + (p >> 2), x1 = x0 + 16;
  const bf16_t* a0 = t + x0 * HD + 8 * (lc ^ swz<HD>(x0)) + sub;
  const bf16_t* a1 = t + x1 * HD + 8 * (lc ^ swz<HD>(x1)) + sub;
  const uint2 v0 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a0));
  const uint2 v1 = __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a1));
  return __builtin_bit_cast(bf16x8, make_uint4(v0.x, v0.y, v1.x, v1.y));
}

// lds_tr_chunk issued as inline assembly. The compiler's wait insertion treats the
// transpose-read builtin as possibly overlapping any direct global->LDS load in flight and
// waits for all of them before it; kernels that keep loads in flight into other buffers
// while they read use this form. The two reads are waited for (lgkmcnt(0)) inside the
// same statement, which also makes every use of the result follow the wait.
template <int HD>
__device__ __forceinline__ bf16x8 lds_tr_chunk_nowait(const bf16_t* t, int k0, int m0, int lane) {
  const int p = lane & 15, j = lane >> 4;
  const int col = m0 + 4 * (p & 3);
  const int lc = col >> 3, sub = col & 7;
  const int x0 = k0 + 4 * j + (p >> 2), x1 = x0 + 16;
  const bf16_t* a0 = t + x0 * HD + 8 * (lc ^ swz<HD>(x0)) + sub;
  const bf16_t* a1 = t + x1 * HD + 8 * (lc ^ swz<HD>(x1)) + sub;
  const uint32_t o0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)a0;
  const uint32_t o1 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)a1;
  uint2 v0, v1;
  asm volatile("ds_read_b64_tr_b16 %0, %2\n\tds_read_b64_tr_b16 %1, %3\n\ts_waitcnt lgkmcnt(0)"
               : "=&v"(v0), "=&v"(v1) : "v"(o0), "v"(o1) : "memory");
  return __builtin_bit_cast(bf16x8, make_uint4(v0.x, v0.y, v1.x, v1.y));
}

// MFMA 16x16x16 A operand of the transposed tile: lane (r = lane % 16, j = lane / 16)
// receives X[k0 + 4j + i][m0 + r], i = 0..3 (one ds_read_b64_tr_b16; addressing as above).
template <int HD>
__device__ __forceinline__ uint2 lds_tr4(const bf16_t* t, int k0, int m0, int lane) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const int p = lane & 15, j = lane >> 4;
  const int col = m0 + 4 * (p & 3);
  const int x0 = k0 + 4 * j + (p >> 2);
  const bf16_t* a0 = t + x0 * HD + 8 * ((col >> 3) ^ swz<HD>(x0)) + (col & 7);
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)a0));
}

// Online-softmax state of one wave over QB blocks of 16 queries.
// Two VALU savings on the hot path: (1) the reference maximum is only raised when a new
// tile maximum exceeds it by more than kRescale (log2 units), so the O accumulators are
// rescaled rarely (probabilities stay <= 2^kRescale, far from f32 overflow); (2) the row
// sums come from the matrix cores: an all-ones A operand in the PV product accumulates
// sum_k P for each query in the same pass as O.
constexpr float kRescale = 8.0f;

template <typename T> __device__ __forceinline__ typename Chunk<T>::type ones_chunk();
template <> __device__ __forceinline__ bf16x8 ones_chunk<bf16_t>() {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)1.0f;
  return r;
}
template <> __device__ __forceinline__ f32x8 ones_chunk<float>() {
  return f32x8{1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
}

// LSE_ONLY: only the softmax statistics (reference maximum and row sums) are formed, in
// exactly the order of the full step, so the log-sum-exp equals the full step's bit for
// bit; the V^T reads and the P V products are skipped and finish() writes no output rows.
// PS (staged steps only): the keys arrive multiplied by the softmax scale times log2(e), so
// a score is already in the exponent's units, and each score MFMA starts from minus the
// reference maximum: its result is the exponent itself, with no multiply-add per score.
// A tile whose maximum raises the reference is shifted once by the rise (shift()).
template <typename T, int HD, int QB, bool LSE_ONLY = false, bool PS = false>
struct WaveAttn {
  static constexpr int NCH = HD / 32;  // chunks of the head dim
  static constexpr int DB = HD / 16;   // 16-wide dim blocks of O^T
  typedef typename Chunk<T>::type CT;
  CT qf[QB][NCH];
  float mx[QB];      // reference maximum (log2 domain, scaled)
  f32x4 o[QB][DB];
  f32x4 lsum[QB];    // row sums (every element holds the same sum)
  f32x4 cneg[QB];    // PS: minus the reference maximum (0 while it is -inf), the scores' start

  __device__ void init() {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      mx[qb] = kNegInf;
      cneg[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
      lsum[qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int db = 0; db < DB; ++db) o[qb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  // Process one tile of KB 16-key blocks (KB even). kfrag(kb, c) gives the A chunk of
  // key block kb, vfrag(db, kp) the A chunk of V^T for dim block db and key pair kp,
  // keyok(kb, i, qb) whether key 4j+i of block kb may be seen by this lane's query.
  // MASKED = false: every key of the tile may be seen by every query (keyok is not called).
  template <int KB, typename KF, typename VF, typename OK, bool MASKED = true>
  __device__ __forceinline__ void tile(float sl2, KF kfrag, VF vfrag, OK keyok) {
    f32x4 s[QB][KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        CT a = kfrag(kb, c);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb][kb] = mma(a, qf[qb][c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : s[qb][kb]);
      }
    // V^T fragments are read now so that their LDS latency hides behind the softmax
    CT vr[DB][KB / 2];
    if constexpr (!LSE_ONLY) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kp = 0; kp < KB / 2; ++kp) vr[db][kp] = vfrag(db, kp);
    }
    CT pf[QB][KB / 2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float tmax = kNegInf;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = !MASKED || keyok(kb, i, qb) ? s[qb][kb][i] : kNegInf;
          s[qb][kb][i] = x;
          tmax = fmaxf(tmax, x);
        }
      tmax = col_max(tmax) * sl2;          // scale > 0 keeps the order
      const bool raise = tmax > mx[qb] + kRescale;
      if (__builtin_amdgcn_ballot_w64(raise)) {   // wave-uniform: rescale only when needed
        const float mnew = raise ? tmax : mx[qb];
        const float alpha = raise ? fast_exp2(mx[qb] - mnew) : 1.0f;
        mx[qb] = mnew;
        lsum[qb] *= alpha;
        if constexpr (!LSE_ONLY) {
#pragma unroll
          for (int db = 0; db < DB; ++db) o[qb][db] *= alpha;
        }
      }
      const float mref = mx[qb] == kNegInf ? 0.f : mx[qb];
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        float v8[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          v8[i] = fast_exp2(__builtin_fmaf(s[qb][2 * kp][i], sl2, -mref));
          v8[4 + i] = fast_exp2(__builtin_fmaf(s[qb][2 * kp + 1][i], sl2, -mref));
        }
        pf[qb][kp] = make_chunk<T>(v8);
      }
    }
    const CT ones = ones_chunk<T>();
#pragma unroll
    for (int kp = 0; kp < KB / 2; ++kp)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) lsum[qb] = mma(ones, pf[qb][kp], lsum[qb]);
    if constexpr (!LSE_ONLY) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kp = 0; kp < KB / 2; ++kp)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][db] = mma(vr[db][kp], pf[qb][kp], o[qb][db]);
    }
  }

  // ---- the step split into its stages, for kernels that software-pipeline key tiles ----
  // Scores S^T of a tile of KB 16-key blocks: s[qb][kb] (this lane: keys 4j + i of block kb
  // for query r of block qb).
  template <int KB, typename KF>
  __device__ __forceinline__ void scores(f32x4 (&s)[QB][KB], KF kfrag) const {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        CT a = kfrag(kb, c);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          s[qb][kb] = mma(a, qf[qb][c], c == 0 ? (PS ? cneg[qb] : f32x4{0.f, 0.f, 0.f, 0.f}) : s[qb][kb]);
      }
  }
  // Masks a score tile (MASK: keyok(kb, i) false -> -inf) and moves the reference maximum:
  // like tile(), it is raised only when the tile's maximum exceeds it by more than
  // kRescale. Returns whether any query of the wave raised it (wave-uniform); alpha[qb] is
  // then the factor for the accumulated O and row sums (1 where not raised), and, PS,
  // delta[qb] the rise of the reference against the one the tile's scores start from (0
  // where not raised), for shift(). Neither is written when it returns false.
  template <int KB, bool MASK, typename OK>
  __device__ __forceinline__ bool tile_max(f32x4 (&s)[QB][KB], float sl2, OK keyok, float (&alpha)[QB],
                                           float (&delta)[QB]) {
    float tloc[QB];
    bool up = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float tmax = kNegInf;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (MASK) s[qb][kb][i] = keyok(kb, i) ? s[qb][kb][i] : kNegInf;
          tmax = fmaxf(tmax, s[qb][kb][i]);
        }
      tloc[qb] = tmax;
      // the test below on this lane's maximum alone: the query's maximum over its four
      // lanes passes it exactly when one of them does (rounding keeps the order)
      up |= (PS ? tmax + -cneg[qb][0] : tmax * sl2) > mx[qb] + kRescale;
    }
    // the usual case once the first tiles are in: no query's reference moves, and the
    // cross-lane maxima, new references and factors are skipped (wave-uniform branch)
    if (__builtin_amdgcn_ballot_w64(up) == 0) return false;
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float cref = -cneg[qb][0];
      const float tmax = PS ? col_max(tloc[qb]) + cref : col_max(tloc[qb]) * sl2;
      const bool raise = tmax > mx[qb] + kRescale;
      const float mnew = raise ? tmax : mx[qb];
      alpha[qb] = raise ? fast_exp2(mx[qb] - mnew) : 1.0f;
      mx[qb] = mnew;
      if constexpr (PS) delta[qb] = raise ? mnew - cref : 0.f;
      any |= __builtin_amdgcn_ballot_w64(raise) != 0;   // no short-circuit: no branch
    }
    return any;
  }
  // PS, after a raise: moves a score tile that started from the previous reference onto
  // the new one, and makes the new one the start of the next tiles' scores
  template <int KB>
  __device__ __forceinline__ void shift(f32x4 (&s)[QB][KB], const float (&delta)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) s[qb][kb][i] -= delta[qb];
      const float c = mx[qb] == kNegInf ? 0.f : -mx[qb];
      cneg[qb] = f32x4{c, c, c, c};
    }
  }
  __device__ __forceinline__ void rescale(const float (&alpha)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      lsum[qb] *= alpha[qb];
      if constexpr (!LSE_ONLY) {
#pragma unroll
        for (int db = 0; db < DB; ++db) o[qb][db] *= alpha[qb];
      }
    }
  }
  // Probabilities of a masked score tile against the current reference maxima, packed as
  // the B operands of the P V product.
  template <int KB>
  __device__ __forceinline__ void probs(const f32x4 (&s)[QB][KB], float sl2, CT (&pf)[QB][KB / 2]) const {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float mref = mx[qb] == kNegInf ? 0.f : mx[qb];
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        float v8[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (PS) {
            v8[i] = fast_exp2(s[qb][2 * kp][i]);
            v8[4 + i] = fast_exp2(s[qb][2 * kp + 1][i]);
          } else {
            v8[i] = fast_exp2(__builtin_fmaf(s[qb][2 * kp][i], sl2, -mref));
            v8[4 + i] = fast_exp2(__builtin_fmaf(s[qb][2 * kp + 1][i], sl2, -mref));
          }
        }
        pf[qb][kp] = make_chunk<T>(v8);
      }
    }
  }
  // Row sums and O += V^T P^T for one tile (vfrag as in tile()).
  template <int KB, typename VF>
  __device__ __forceinline__ void pv(const CT (&pf)[QB][KB / 2], VF vfrag) {
    const CT ones = ones_chunk<T>();
#pragma unroll
    for (int kp = 0; kp < KB / 2; ++kp)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) lsum[qb] = mma(ones, pf[qb][kp], lsum[qb]);
    if constexpr (!LSE_ONLY) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kp = 0; kp < KB / 2; ++kp) {
          const CT vr = vfrag(db, kp);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) o[qb][db] = mma(vr, pf[qb][kp], o[qb][db]);
        }
    }
  }

  // Normalise and store O rows (query q0 + 16 qb + r) and natural-log LSE.
  // out: rows in the storage type, or float32 where a caller needs the unrounded output
  template <typename OT>
  __device__ void finish(int lane, long long row0, OT* out, float* lse, const uint8_t* qvalid, int qidx0) {
    const int r = lane & 15, j = lane >> 4;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float l = lsum[qb][0];
      const bool qok = qvalid == nullptr || qvalid[qidx0 + 16 * qb + r];
      const bool any = qok && l > 0.f;
      const float inv = any ? 1.0f / l : 0.f;
      const long long row = row0 + 16 * qb + r;
      if constexpr (!LSE_ONLY) {
#pragma unroll
        for (int db = 0; db < DB; ++db) store4(out + row * HD + 16 * db + 4 * j, o[qb][db], inv);
      }
      if (j == 0) lse[row] = any ? (mx[qb] + log2f(l)) * kLn2 : kNegInf;
    }
  }
};

template <typename T, int HD, int QB, bool LO, bool PS>
__device__ __forceinline__ void load_q(WaveAttn<T, HD, QB, LO, PS>& w, const T* qrow0, int lane) {
  const int r = lane & 15, j = lane >> 4;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int c = 0; c < WaveAttn<T, HD, QB, LO, PS>::NCH; ++c)
      w.qf[qb][c] = load_chunk(qrow0 + (size_t)(16 * qb + r) * HD + 32 * c + 8 * j);
}


}  // namespace
}  // namespace bsa
