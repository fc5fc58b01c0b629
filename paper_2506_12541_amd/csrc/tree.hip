// Ball-tree ordering of point clouds (the ordering Ball Tree Attention runs on,
// Section 2.1 and 2.2), and the row gather/scatter between point order and ball order.
//
// Construction: a node of capacity C holding the point set S splits on the axis of
// largest spread (float64 difference of float32 extremes, lowest axis on ties); its
// points ordered by (coordinate, index) are cut after ceil(|S|/2): left child in slots
// [0, C/2), right child in [C/2, C). The result depends only on node sets, so the GPU
// is free to use any partition that preserves them.
//
// GPU plan. The three per-axis orderings of every cloud are produced once by a stable
// LSD radix sort (4-bit digits). Each node then keeps, for every axis, its points
// sorted on that axis, stored at the node's own slot range. A split reads the extremes
// of each axis at the ends of the lists and the median at position ceil(n/2)-1 of the
// split axis; every list is then stably partitioned by "key <= median key", which keeps
// all three lists sorted in both children. Levels with nodes larger than 1024 slots run
// as three small kernels per level over all nodes; the last ten levels run inside one
// workgroup per 1024-slot node, entirely in LDS.
#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortItems = 8;
constexpr int kSortTile = kSortThreads * kSortItems;  // 2048 keys per workgroup
constexpr int kPartTile = 2048;                       // slots per partition workgroup
constexpr int kBottom = 1024;                         // node size finished in LDS

__device__ __forceinline__ uint32_t ordered_key(float x) {
  x = x + 0.0f;  // -0.0 -> +0.0
  uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Real points in the node with index `node` among the nodes of capacity 2^log2c of one
// cloud: follow the root-to-node path, left children take the ceiling half.
__device__ __forceinline__ int node_count(int n_real, int log2_npad, int log2c, int node) {
  int cnt = n_real;
  for (int t = log2_npad - log2c - 1; t >= 0; --t)
    cnt = ((node >> t) & 1) ? (cnt >> 1) : ((cnt + 1) >> 1);
  return cnt;
}

__device__ __forceinline__ float coord(const float* pts, int dim, int g, int a) {
  return a < dim ? pts[(size_t)g * dim + a] : 0.0f;
}

// Block-wide exclusive scan of one value per thread (blockDim.x threads, <= 1024).
__device__ int block_exclusive_scan(int v, int* lds_tmp, int* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds_tmp[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) { int t = lds_tmp[w]; lds_tmp[w] = run; run += t; }
    lds_tmp[nw] = run;
  }
  __syncthreads();
  int res = x - v + lds_tmp[wid];
  if (total) *total = lds_tmp[nw];
  __syncthreads();
  return res;
}

// ---- radix sort of (key, point) per axis; grid.y = axis ----
__global__ void __launch_bounds__(kSortThreads) sort_init_kernel(const float* pts, int dim, int m,
                                                                 uint32_t* keys, uint32_t* vals) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  int a = blockIdx.y;
  if (i >= m) return;
  keys[(size_t)a * m + i] = ordered_key(coord(pts, dim, i, a));
  vals[(size_t)a * m + i] = (uint32_t)i;
}

__device__ __forceinline__ uint32_t sort_digit(uint32_t key, uint32_t val, int pass, int n_real) {
  return pass < 8 ? (key >> (4 * pass)) & 15u : ((val / (uint32_t)n_real) >> (4 * (pass - 8))) & 15u;
}

__global__ void __launch_bounds__(kSortThreads) sort_hist_kernel(const uint32_t* keys, const uint32_t* vals,
                                                                 int m, int pass, int n_real, int ntiles,
                                                                 uint32_t* hist) {
  __shared__ uint32_t cnt[16];
  const int a = blockIdx.y, tile = blockIdx.x;
  if (threadIdx.x < 16) cnt[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t* K = keys + (size_t)a * m;
  const uint32_t* V = vals + (size_t)a * m;
  for (int it = 0; it < kSortItems; ++it) {
    int i = tile * kSortTile + it * kSortThreads + threadIdx.x;
    if (i < m) atomicAdd(&cnt[sort_digit(K[i], V[i], pass, n_real)], 1u);
  }
  __syncthreads();
  if (threadIdx.x < 16) hist[((size_t)a * 16 + threadIdx.x) * ntiles + tile] = cnt[threadIdx.x];
}

// Exclusive scan of hist[a] in digit-major order; one 1024-thread workgroup per axis.
__global__ void __launch_bounds__(1024) sort_scan_kernel(uint32_t* hist, int ntiles) {
  __shared__ int tmp[17];
  uint32_t* H = hist + (size_t)blockIdx.y * 16 * ntiles;
  const int total = 16 * ntiles;
  const int per = (total + 1023) / 1024;
  const int s = threadIdx.x * per;
  int sum = 0;
  for (int i = s; i < s + per && i < total; ++i) sum += (int)H[i];
  int run = block_exclusive_scan(sum, tmp, nullptr);
  for (int i = s; i < s + per && i < total; ++i) {
    int t = (int)H[i];
    H[i] = (uint32_t)run;
    run += t;
  }
}

__global__ void __launch_bounds__(kSortThreads) sort_scatter_kernel(const uint32_t* keys, const uint32_t* vals,
                                                                    uint32_t* keys_out, uint32_t* vals_out,
                                                                    int m, int pass, int n_real, int ntiles,
                                                                    const uint32_t* hist) {
  __shared__ int cnt[16 * kSortThreads];  // digit-major: cnt[d * 256 + thread]
  __shared__ int tmp[8];
  const int a = blockIdx.y, tile = blockIdx.x, t = threadIdx.x;
  const uint32_t* K = keys + (size_t)a * m;
  const uint32_t* V = vals + (size_t)a * m;
  uint32_t k[kSortItems], v[kSortItems];
  int dg[kSortItems];
  int mine[16];
#pragma unroll
  for (int d = 0; d < 16; ++d) mine[d] = 0;
  const int base_i = tile * kSortTile + t * kSortItems;  // consecutive items per thread
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    int i = base_i + it;
    dg[it] = -1;
    if (i < m) {
      k[it] = K[i];
      v[it] = V[i];
      dg[it] = (int)sort_digit(k[it], v[it], pass, n_real);
#pragma unroll
      for (int d = 0; d < 16; ++d) mine[d] += (dg[it] == d);
    }
  }
#pragma unroll
  for (int d = 0; d < 16; ++d) cnt[d * kSortThreads + t] = mine[d];
  __syncthreads();
  // scan 4096 digit-major entries: thread t owns entries [16t, 16t+16)
  int loc[16];
  int sum = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) { loc[e] = cnt[16 * t + e]; sum += loc[e]; }
  int run = block_exclusive_scan(sum, tmp, nullptr);
#pragma unroll
  for (int e = 0; e < 16; ++e) { int x = loc[e]; cnt[16 * t + e] = run; run += x; }
  __syncthreads();
  // digit offsets within the tile: entry (d, thread 0) holds the start of digit d
  int pos[16];
  const uint32_t* H = hist + (size_t)a * 16 * ntiles;
#pragma unroll
  for (int d = 0; d < 16; ++d)
    pos[d] = (int)H[(size_t)d * ntiles + tile] + cnt[d * kSortThreads + t] - cnt[d * kSortThreads];
  uint32_t* KO = keys_out + (size_t)a * m;
  uint32_t* VO = vals_out + (size_t)a * m;
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    if (dg[it] < 0) continue;
    int p = 0;
#pragma unroll
    for (int d = 0; d < 16; ++d)
      if (dg[it] == d) p = pos[d]++;
    KO[p] = k[it];
    VO[p] = v[it];
  }
}

// Sorted position -> the axis list of its cloud, at slots [b*n_pad, b*n_pad + n_real).
__global__ void lists_init_kernel(const uint32_t* vals, int m, int n_real, int n_pad, int batch,
                                  int* lists) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int a = blockIdx.y;
  const size_t slots = (size_t)batch * n_pad;
  if (i >= slots) return;
  int b = (int)(i / n_pad), r = (int)(i % n_pad);
  lists[a * slots + i] = r < n_real ? (int)vals[(size_t)a * m + (size_t)b * n_real + r] : -1;
}

// ---- one top level: nodes of capacity 2^log2c (> kBottom) ----
struct NodeSplit {
  int axis;
  int med_idx;
  float med;
  int cnt;
};

__global__ void node_split_kernel(const float* pts, int dim, int n_real, int n_pad, int log2_npad,
                                  int log2c, int nodes, const int* lists, NodeSplit* out) {
  int nd = blockIdx.x * blockDim.x + threadIdx.x;
  if (nd >= nodes) return;
  const size_t slots = (size_t)(nodes) << log2c;
  const int per_cloud = n_pad >> log2c;
  int cnt = node_count(n_real, log2_npad, log2c, nd % per_cloud);
  size_t start = (size_t)nd << log2c;
  NodeSplit s{0, -1, 0.0f, cnt};
  if (cnt > 0) {
    double best = -1.0;
    for (int a = 0; a < 3; ++a) {
      float lo = coord(pts, dim, lists[a * slots + start], a);
      float hi = coord(pts, dim, lists[a * slots + start + cnt - 1], a);
      double sp = (double)hi - (double)lo;
      if (sp > best) { best = sp; s.axis = a; }
    }
    s.med_idx = lists[s.axis * slots + start + (cnt + 1) / 2 - 1];
    s.med = coord(pts, dim, s.med_idx, s.axis);
  }
  out[nd] = s;
}

__device__ __forceinline__ bool goes_left(const float* pts, int dim, int g, const NodeSplit& s) {
  float c = coord(pts, dim, g, s.axis);
  return c < s.med || (c == s.med && g <= s.med_idx);
}

__global__ void __launch_bounds__(256) part_count_kernel(const float* pts, int dim, int log2c, const int* lists,
                                                         const NodeSplit* splits, int tiles_per_list,
                                                         int* tilecnt) {
  __shared__ int tmp[8];
  const int a = blockIdx.y, tile = blockIdx.x;
  const size_t slots = (size_t)tiles_per_list * kPartTile;
  const size_t s0 = (size_t)tile * kPartTile;
  const int nd = (int)(s0 >> log2c);
  NodeSplit sp = splits[nd];
  const int off = (int)(s0 - ((size_t)nd << log2c));
  int c = 0;
  for (int i = threadIdx.x; i < kPartTile; i += 256) {
    if (off + i < sp.cnt) c += goes_left(pts, dim, lists[a * slots + s0 + i], sp);
  }
  int total;
  block_exclusive_scan(c, tmp, &total);
  if (threadIdx.x == 0) tilecnt[a * tiles_per_list + tile] = total;
}

__global__ void __launch_bounds__(256) part_scatter_kernel(const float* pts, int dim, int log2c,
                                                           const int* lists, int* lists_out,
                                                           const NodeSplit* splits, int tiles_per_list,
                                                           const int* tilecnt) {
  __shared__ int tmp[8];
  const int a = blockIdx.y, tile = blockIdx.x;
  const size_t slots = (size_t)tiles_per_list * kPartTile;
  const size_t s0 = (size_t)tile * kPartTile;
  const int nd = (int)(s0 >> log2c);
  const NodeSplit sp = splits[nd];
  const size_t node_start = (size_t)nd << log2c;
  const int off = (int)(s0 - node_start);
  const int first_tile = (int)(node_start / kPartTile);
  // left-going elements in earlier tiles of this node
  int before = 0;
  for (int t = first_tile + (int)threadIdx.x; t < tile; t += 256) before += tilecnt[a * tiles_per_list + t];
  int left_before;
  block_exclusive_scan(before, tmp, &left_before);
  // each thread handles 8 consecutive slots
  constexpr int kItems = kPartTile / 256;
  int g[kItems];
  int f[kItems];
  int mine = 0;
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    int i = threadIdx.x * kItems + it;
    f[it] = -1;
    if (off + i < sp.cnt) {
      g[it] = lists[a * slots + s0 + i];
      f[it] = goes_left(pts, dim, g[it], sp) ? 1 : 0;
      mine += f[it];
    }
  }
  int lrank = block_exclusive_scan(mine, tmp, nullptr) + left_before;
  const int half = 1 << (log2c - 1);
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    if (f[it] < 0) continue;
    int pos_in_node = off + threadIdx.x * kItems + it;
    size_t dst;
    if (f[it]) {
      dst = node_start + lrank;
      ++lrank;
    } else {
      dst = node_start + half + (pos_in_node - lrank);
    }
    lists_out[a * slots + dst] = g[it];
  }
}

// ---- the last levels of one node of capacity T <= 1024, in LDS ----
__global__ void __launch_bounds__(256) bottom_kernel(const float* pts, int dim, int n_real, int n_pad,
                                                     int log2_npad, int log2t, int nodes, const int* lists,
                                                     int* perm) {
  __shared__ float4 el[3 * kBottom];   // (x, y, z, point as int bits) per list slot
  __shared__ int sub_axis[kBottom / 2];
  __shared__ int sub_idx[kBottom / 2];
  __shared__ float sub_med[kBottom / 2];
  __shared__ int tmp[8];
  const int T = 1 << log2t;
  const int nd = blockIdx.x;
  const size_t slots = (size_t)nodes << log2t;
  const size_t start = (size_t)nd << log2t;
  const int per_cloud = n_pad >> log2t;
  const int node_in_cloud = nd % per_cloud;
  const int cloud = nd / per_cloud;
  const int cnt0 = node_count(n_real, log2_npad, log2t, node_in_cloud);
  for (int i = threadIdx.x; i < 3 * T; i += 256) {
    int a = i / T, r = i % T;
    float4 e = make_float4(0.f, 0.f, 0.f, __int_as_float(-1));
    if (r < cnt0) {
      int g = lists[a * slots + start + r];
      e = make_float4(coord(pts, dim, g, 0), coord(pts, dim, g, 1), coord(pts, dim, g, 2), __int_as_float(g));
    }
    el[i] = e;
  }
  __syncthreads();
  const int items = (3 * T + 255) / 256;  // <= 12
  for (int log2c = log2t; log2c >= 1; --log2c) {
    const int C = 1 << log2c;
    const int nsub = T >> log2c;
    // split of every sub-node
    for (int s = threadIdx.x; s < nsub; s += 256) {
      int cnt = node_count(n_real, log2_npad, log2c, node_in_cloud * nsub + s);
      int axis = 0, midx = -1;
      float med = 0.f;
      if (cnt > 0) {
        double best = -1.0;
        for (int a = 0; a < 3; ++a) {
          float4 lo = el[a * T + s * C], hi = el[a * T + s * C + cnt - 1];
          float l = a == 0 ? lo.x : (a == 1 ? lo.y : lo.z);
          float h = a == 0 ? hi.x : (a == 1 ? hi.y : hi.z);
          double sp = (double)h - (double)l;
          if (sp > best) { best = sp; axis = a; }
        }
        float4 me = el[axis * T + s * C + (cnt + 1) / 2 - 1];
        med = axis == 0 ? me.x : (axis == 1 ? me.y : me.z);
        midx = __float_as_int(me.w);
      }
      sub_axis[s] = axis;
      sub_idx[s] = midx;
      sub_med[s] = med;
    }
    __syncthreads();
    float4 e[12];
    int f[12];
    int mine = 0;
#pragma unroll
    for (int it = 0; it < 12; ++it) {
      f[it] = -1;
      int i = threadIdx.x * items + it;
      if (it < items && i < 3 * T) {
        e[it] = el[i];
        int g = __float_as_int(e[it].w);
        if (g >= 0) {
          int s = (i % T) >> log2c;
          int ax = sub_axis[s];
          float c = ax == 0 ? e[it].x : (ax == 1 ? e[it].y : e[it].z);
          f[it] = (c < sub_med[s] || (c == sub_med[s] && g <= sub_idx[s])) ? 1 : 0;
          mine += f[it];
        }
      }
    }
    // exclusive prefix of left flags over the concatenated lists; sub-node starts are
    // aligned to C, so the prefix at a sub-node start is subtracted below
    int pre = block_exclusive_scan(mine, tmp, nullptr);
    __shared__ int start_pref[3 * kBottom / 2];
    // record prefix at each sub-node start: the thread owning index (s*C) writes it
    {
      int run = pre;
#pragma unroll
      for (int it = 0; it < 12; ++it) {
        int i = threadIdx.x * items + it;
        if (it < items && i < 3 * T) {
          if ((i & (C - 1)) == 0) start_pref[i >> log2c] = run;
          run += f[it] > 0 ? 1 : 0;
        }
      }
    }
    __syncthreads();
    // all old values are in registers: rewrite the lists in place
    for (int i = threadIdx.x; i < 3 * T; i += 256) el[i] = make_float4(0.f, 0.f, 0.f, __int_as_float(-1));
    __syncthreads();
    {
      int run = pre;
#pragma unroll
      for (int it = 0; it < 12; ++it) {
        int i = threadIdx.x * items + it;
        if (it < items && i < 3 * T && f[it] >= 0) {
          int sub_start = i & ~(C - 1);
          int lr = run - start_pref[i >> log2c];   // left flags before i in this sub-node
          int pos = i - sub_start;
          int dst = f[it] ? sub_start + lr : sub_start + C / 2 + (pos - lr);
          el[dst] = e[it];
        }
        if (it < items && i < 3 * T) run += f[it] > 0 ? 1 : 0;
      }
    }
    __syncthreads();
  }
  for (int r = threadIdx.x; r < T; r += 256) {
    int g = __float_as_int(el[r].w);
    perm[start + r] = g >= 0 ? g - cloud * n_real : -1;
  }
}

// ---- row gather / scatter between point order and ball order ----
template <typename T>
__global__ void permute_kernel(const T* src, const int* perm, int n_real, int n_pad, int heads, int hd,
                               T* dst, uint8_t* valid, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  // dst index [b, h, s, c]
  int c = (int)(i % hd);
  size_t r = i / hd;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  T val = T(0);
  if (p >= 0) val = src[((size_t)b * n_real + p) * heads * hd + (size_t)h * hd + c];
  dst[i] = val;
  if (valid && h == 0 && c == 0) valid[(size_t)b * n_pad + s] = p >= 0;
}

template <typename T>
__global__ void unpermute_kernel(const T* src, const int* perm, int n_real, int n_pad, int heads, int hd,
                                 T* dst, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % hd);
  size_t r = i / hd;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  if (p >= 0) dst[((size_t)b * n_real + p) * heads * hd + (size_t)h * hd + c] = src[i];
}

// 16-byte variant: one work item moves one 16-byte piece of a head row.
__global__ void permute16_kernel(const uint4* src, const int* perm, int n_real, int n_pad, int heads, int vpr,
                                 uint4* dst, uint8_t* valid, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % vpr);
  size_t r = i / vpr;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  uint4 val = make_uint4(0, 0, 0, 0);
  if (p >= 0) val = src[((size_t)b * n_real + p) * heads * vpr + (size_t)h * vpr + c];
  dst[i] = val;
  if (valid && h == 0 && c == 0) valid[(size_t)b * n_pad + s] = p >= 0;
}

__global__ void unpermute16_kernel(const uint4* src, const int* perm, int n_real, int n_pad, int heads, int vpr,
                                   uint4* dst, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % vpr);
  size_t r = i / vpr;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  if (p >= 0) dst[((size_t)b * n_real + p) * heads * vpr + (size_t)h * vpr + c] = src[i];
}

inline int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

}  // namespace

size_t tree_workspace_bytes(int64_t n_real, int64_t n_pad, int batch) {
  const size_t m = (size_t)batch * n_real;
  const size_t slots = (size_t)batch * n_pad;
  const size_t ntiles = (m + kSortTile - 1) / kSortTile;
  size_t b = 0;
  auto add = [&](size_t x) { b += (x + 255) & ~size_t(255); };
  add(4 * 3 * m);          // keys a
  add(4 * 3 * m);          // keys b
  add(4 * 3 * m);          // vals a
  add(4 * 3 * m);          // vals b
  add(4 * 3 * 16 * ntiles);  // histograms
  add(4 * 3 * slots);      // lists a
  add(4 * 3 * slots);      // lists b
  add(sizeof(NodeSplit) * (slots / 2 + 1));
  add(4 * 3 * (slots / kPartTile + 1));
  return b;
}

hipError_t launch_build_tree(const float* pts, int64_t n_real, int dim, int64_t n_pad, int batch,
                             int* perm, void* ws, hipStream_t st) {
  const size_t m = (size_t)batch * n_real;
  const size_t slots = (size_t)batch * n_pad;
  const int ntiles = (int)((m + kSortTile - 1) / kSortTile);
  char* p = (char*)ws;
  auto take = [&](size_t x) { char* r = p; p += (x + 255) & ~size_t(255); return r; };
  uint32_t* ka = (uint32_t*)take(4 * 3 * m);
  uint32_t* kb = (uint32_t*)take(4 * 3 * m);
  uint32_t* va = (uint32_t*)take(4 * 3 * m);
  uint32_t* vb = (uint32_t*)take(4 * 3 * m);
  uint32_t* hist = (uint32_t*)take(4 * 3 * 16 * (size_t)ntiles);
  int* la = (int*)take(4 * 3 * slots);
  int* lb = (int*)take(4 * 3 * slots);
  NodeSplit* splits = (NodeSplit*)take(sizeof(NodeSplit) * (slots / 2 + 1));
  int* tilecnt = (int*)take(4 * 3 * (slots / kPartTile + 1));

  hipLaunchKernelGGL(sort_init_kernel, dim3((unsigned)((m + 255) / 256), 3), dim3(256), 0, st, pts, dim,
                     (int)m, ka, va);
  int passes = 8;
  for (int bits = 0; (1 << bits) < batch; bits += 4) ++passes;
  for (int pass = 0; pass < passes; ++pass) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3(ntiles, 3), dim3(kSortThreads), 0, st, ka, va, (int)m, pass,
                       (int)n_real, ntiles, hist);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(1, 3), dim3(1024), 0, st, hist, ntiles);
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(ntiles, 3), dim3(kSortThreads), 0, st, ka, va, kb, vb,
                       (int)m, pass, (int)n_real, ntiles, hist);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  hipLaunchKernelGGL(lists_init_kernel, dim3((unsigned)((slots + 255) / 256), 3), dim3(256), 0, st, va,
                     (int)m, (int)n_real, (int)n_pad, batch, la);
  const int log2_npad = ilog2(n_pad);
  const int log2t = log2_npad < 10 ? log2_npad : 10;
  for (int log2c = log2_npad; log2c > log2t; --log2c) {
    const int nodes = (int)(slots >> log2c);
    const int tiles = (int)(slots / kPartTile);
    hipLaunchKernelGGL(node_split_kernel, dim3((nodes + 63) / 64), dim3(64), 0, st, pts, dim, (int)n_real,
                       (int)n_pad, log2_npad, log2c, nodes, la, splits);
    hipLaunchKernelGGL(part_count_kernel, dim3(tiles, 3), dim3(256), 0, st, pts, dim, log2c, la, splits,
                       tiles, tilecnt);
    hipLaunchKernelGGL(part_scatter_kernel, dim3(tiles, 3), dim3(256), 0, st, pts, dim, log2c, la, lb,
                       splits, tiles, tilecnt);
    std::swap(la, lb);
  }
  const int nodes = (int)(slots >> log2t);
  hipLaunchKernelGGL(bottom_kernel, dim3(nodes), dim3(256), 0, st, pts, dim, (int)n_real, (int)n_pad,
                     log2_npad, log2t, nodes, la, perm);
  return hipGetLastError();
}

size_t radix_sort_hist_words(long long n) { return (size_t)16 * ((n + kSortTile - 1) / kSortTile); }

hipError_t launch_radix_sort_pairs(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                                   uint32_t* hist, long long n, int bits, uint32_t** keys_out, uint32_t** vals_out,
                                   hipStream_t st) {
  const int ntiles = (int)((n + kSortTile - 1) / kSortTile);
  const int passes = (bits + 3) / 4;  // key digits only (pass < 8)
  uint32_t *ka = keys, *va = vals, *kb = keys_tmp, *vb = vals_tmp;
  for (int pass = 0; pass < passes; ++pass) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3(ntiles, 1), dim3(kSortThreads), 0, st, ka, va, (int)n, pass, 1, ntiles,
                       hist);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(1, 1), dim3(1024), 0, st, hist, ntiles);
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(ntiles, 1), dim3(kSortThreads), 0, st, ka, va, kb, vb, (int)n, pass,
                       1, ntiles, hist);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  *keys_out = ka;
  *vals_out = va;
  return hipGetLastError();
}

hipError_t launch_permute(const void* src, const int* perm, int64_t n_real, int64_t n_pad, int batch,
                          int heads, int hd, int dtype, void* dst, uint8_t* valid, bool inverse,
                          hipStream_t st) {
  const size_t esz = dtype == 0 ? 4 : 2;
  if ((hd * esz) % 16 == 0) {
    const int vpr = (int)(hd * esz / 16);
    const size_t total = (size_t)batch * heads * n_pad * vpr;
    const unsigned blocks = (unsigned)((total + 255) / 256);
    if (!inverse)
      hipLaunchKernelGGL(permute16_kernel, dim3(blocks), dim3(256), 0, st, (const uint4*)src, perm, (int)n_real,
                         (int)n_pad, heads, vpr, (uint4*)dst, valid, total);
    else
      hipLaunchKernelGGL(unpermute16_kernel, dim3(blocks), dim3(256), 0, st, (const uint4*)src, perm, (int)n_real,
                         (int)n_pad, heads, vpr, (uint4*)dst, total);
    return hipGetLastError();
  }
  const size_t total = (size_t)batch * heads * n_pad * hd;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  if (!inverse) {
    if (dtype == 0)
      hipLaunchKernelGGL(permute_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (float*)dst, valid, total);
    else
      hipLaunchKernelGGL(permute_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, (const uint16_t*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (uint16_t*)dst, valid, total);
  } else {
    if (dtype == 0)
      hipLaunchKernelGGL(unpermute_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (float*)dst, total);
    else
      hipLaunchKernelGGL(unpermute_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, (const uint16_t*)src,
                         perm, (int)n_real, (int)n_pad, heads, hd, (uint16_t*)dst, total);
  }
  return hipGetLastError();
}

}  // namespace bsa
