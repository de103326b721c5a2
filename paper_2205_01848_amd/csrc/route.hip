// Load counting, capacities, slot assignment + dispatch (GroupBy with the
// Section 4.1 capacity/drop rule), combine (Aggregate) and their backward.
//
// Slot assignment is a stable counting sort of the T*k assignments in
// priority order q = j*T + t (all first choices in token order, then all
// second choices, ...):
//   1. per-chunk expert histograms (4096 assignments per workgroup),
//   2. one workgroup scans them into per-chunk bases and applies capacity,
//   3. each chunk re-ranks its assignments with wavefront ballots (expert id
//      equality masks from 6 ballots, rank = popcount below the lane),
//      giving pos, keep, dest_row and src - all integer, bit-exact.
// The row copies (dispatch gather, combine, their backward) are token-major:
// one wavefront per token, 16-byte vector loads/stores along the row, so x
// is read once even when k rows are written.

#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "validate.hpp"

namespace moe {
namespace {

constexpr int kChunk = 1024;  // assignments per workgroup in the routing kernels

// Is assignment (t, j) live?  Sets status bits when `status` is non-null.
__device__ __forceinline__ bool live_assignment(const int32_t* __restrict__ ids, int t,
                                                int j, int k, int E, int32_t* status) {
  const int32_t* row = ids + static_cast<size_t>(t) * k;
  const int e = row[j];
  if (e < 0 || e >= E) {
    if (status) atomicOr(status, MOE_STATUS_BAD_ID);
    return false;
  }
  for (int jj = 0; jj < j; ++jj) {
    if (row[jj] == e) {
      if (status) atomicOr(status, MOE_STATUS_DUP_ID);
      return false;
    }
  }
  return true;
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

// counts[e] += live assignments of this block's chunk (counts zeroed before)
__global__ __launch_bounds__(256) void count_kernel(const int32_t* __restrict__ ids, int T,
                                                    int E, int k, int32_t* counts,
                                                    int32_t* status) {
  __shared__ int h[kMaxE];
  if (threadIdx.x < kMaxE) h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t n = static_cast<int64_t>(T) * k;
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kChunk;
  const int64_t q1 = min(n, q0 + kChunk);
  for (int64_t q = q0 + threadIdx.x; q < q1; q += 256) {
    const int j = static_cast<int>(q / T), t = static_cast<int>(q - static_cast<int64_t>(j) * T);
    if (live_assignment(ids, t, j, k, E, status)) atomicAdd(&h[ids[static_cast<size_t>(t) * k + j]], 1);
  }
  __syncthreads();
  if (threadIdx.x < E && h[threadIdx.x]) atomicAdd(&counts[threadIdx.x], h[threadIdx.x]);
}

// Eq. 4 / dynamic capacity factors, exact 64-bit integer ceil, + offsets:
// expert e's region starts at the sum of the earlier capacities, each
// rounded up to a multiple of row_align rows.
__global__ __launch_bounds__(64) void capacity_kernel(int T, int k, int E,
                                                      const int32_t* __restrict__ counts,
                                                      int num, int den, int cap_min,
                                                      int row_align,
                                                      int32_t* __restrict__ capacity,
                                                      int32_t* __restrict__ offsets) {
  __shared__ int64_t c[kMaxE];
  const int e = threadIdx.x;
  if (e < E) {
    int64_t v;
    if (counts) {
      const int64_t cnt = max(counts[e], 0);
      v = (static_cast<int64_t>(num) * cnt + den - 1) / den;
    } else {
      v = (static_cast<int64_t>(num) * T * k + static_cast<int64_t>(den) * E - 1) /
          (static_cast<int64_t>(den) * E);
    }
    v = max(v, static_cast<int64_t>(cap_min));
    v = min(v, static_cast<int64_t>(T));
    c[e] = v;
    capacity[e] = static_cast<int32_t>(v);
  }
  __syncthreads();
  if (e == 0) {
    int64_t run = 0;
    for (int i = 0; i < E; ++i) {
      offsets[i] = static_cast<int32_t>(run);
      run += (c[i] + row_align - 1) / row_align * row_align;
    }
    offsets[E] = static_cast<int32_t>(run);
  }
}

// Dispatch step 1: chunk histograms; also initialises src[] to -1.
__global__ __launch_bounds__(256) void route_hist_kernel(
    const int32_t* __restrict__ ids, int T, int E, int k, int nblk, int64_t rows_alloc,
    int32_t* __restrict__ hist, int32_t* __restrict__ src, int32_t* status) {
  __shared__ int h[kMaxE];
  if (threadIdx.x < kMaxE) h[threadIdx.x] = 0;
  const int64_t rs = (rows_alloc + nblk - 1) / nblk;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rs;
  const int64_t r1 = min(rows_alloc, r0 + rs);
  for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) src[r] = -1;
  __syncthreads();
  const int64_t n = static_cast<int64_t>(T) * k;
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kChunk;
  const int64_t q1 = min(n, q0 + kChunk);
  for (int64_t q = q0 + threadIdx.x; q < q1; q += 256) {
    const int j = static_cast<int>(q / T), t = static_cast<int>(q - static_cast<int64_t>(j) * T);
    if (live_assignment(ids, t, j, k, E, status)) atomicAdd(&h[ids[static_cast<size_t>(t) * k + j]], 1);
  }
  __syncthreads();
  if (threadIdx.x < E) hist[static_cast<size_t>(blockIdx.x) * E + threadIdx.x] = h[threadIdx.x];
}

// Usable rows of expert e's region: its capacity, clamped to the region the
// offsets give it and to rows_alloc (0 for a region starting out of range).
__device__ __forceinline__ int64_t region_room(const int32_t* __restrict__ capacity,
                                               const int32_t* __restrict__ offsets,
                                               int64_t rows_alloc, int e) {
  const int64_t off = offsets[e];
  int64_t room = 0;
  if (off >= 0) {
    room = capacity[e];
    room = min(room, static_cast<int64_t>(offsets[e + 1]) - off);
    room = min(room, rows_alloc - off);
    room = max(room, int64_t(0));
  }
  return room;
}

// Dispatch step 2: per-expert exclusive scan over chunks, counts, the usable
// capacity of each region, fill.
__global__ __launch_bounds__(64) void route_scan_kernel(
    const int32_t* __restrict__ hist, int nblk, int E, const int32_t* __restrict__ capacity,
    const int32_t* __restrict__ offsets, int64_t rows_alloc, int32_t* __restrict__ base,
    int32_t* __restrict__ cap_eff, int32_t* __restrict__ counts, int32_t* __restrict__ fill,
    int32_t* status) {
  const int e = threadIdx.x;
  if (e >= E) return;
  int run = 0;
  int b = 0;
  for (; b + 8 <= nblk; b += 8) {   // loads of 8 chunks issued before their adds
    int h[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) h[u] = hist[static_cast<size_t>(b + u) * E + e];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      base[static_cast<size_t>(b + u) * E + e] = run;
      run += h[u];
    }
  }
  for (; b < nblk; ++b) {
    base[static_cast<size_t>(b) * E + e] = run;
    run += hist[static_cast<size_t>(b) * E + e];
  }
  counts[e] = run;
  const int64_t room = region_room(capacity, offsets, rows_alloc, e);
  if (room < capacity[e]) atomicOr(status, MOE_STATUS_REGION);
  cap_eff[e] = static_cast<int32_t>(room);
  fill[e] = static_cast<int32_t>(min(static_cast<int64_t>(run), room));
}

// Dispatch step 3: rank within chunk (wavefront ballots), keep/dest/src.
// SCAN: small batches (at most kScanChunks chunks) skip step 2; every
// workgroup sums the histograms of the chunks before its own, and workgroup
// 0 writes counts, fill and the region status bit.
constexpr int kScanChunks = 64;
template <bool SCAN>
__global__ __launch_bounds__(256) void route_rank_kernel(
    const int32_t* __restrict__ ids, int T, int E, int k, const int32_t* __restrict__ base,
    const int32_t* __restrict__ cap_eff, const int32_t* __restrict__ offsets,
    int32_t* __restrict__ dest_row, int32_t* __restrict__ src,
    const int32_t* __restrict__ hist, int nblk, const int32_t* __restrict__ capacity,
    int64_t rows_alloc, int32_t* __restrict__ counts, int32_t* __restrict__ fill,
    int32_t* status) {
  __shared__ int run[kMaxE];
  __shared__ int wcnt[4][kMaxE];
  __shared__ int capv[kMaxE];
  __shared__ int offv[kMaxE];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if constexpr (SCAN) {
    // wave w sums chunks w, w + 4, ...: those before this one (wcnt) and
    // all of them (tot)
    __shared__ int tot[4][kMaxE];
    if (lane < E) {
      int lo = 0, all = 0;
      for (int b = wave; b < nblk; b += 4) {
        const int v = hist[static_cast<size_t>(b) * E + lane];
        all += v;
        lo += b < static_cast<int>(blockIdx.x) ? v : 0;
      }
      wcnt[wave][lane] = lo;
      tot[wave][lane] = all;
    }
    __syncthreads();
    if (threadIdx.x < E) {
      const int e = threadIdx.x;
      run[e] = wcnt[0][e] + wcnt[1][e] + wcnt[2][e] + wcnt[3][e];
      const int total = tot[0][e] + tot[1][e] + tot[2][e] + tot[3][e];
      const int64_t room = region_room(capacity, offsets, rows_alloc, e);
      if (blockIdx.x == 0) {
        counts[e] = total;
        fill[e] = static_cast<int32_t>(min(static_cast<int64_t>(total), room));
        if (room < capacity[e]) atomicOr(status, MOE_STATUS_REGION);
      }
      capv[e] = static_cast<int32_t>(room);
      offv[e] = offsets[e];
    }
  } else {
    if (threadIdx.x < E) {
      run[threadIdx.x] = base[static_cast<size_t>(blockIdx.x) * E + threadIdx.x];
      capv[threadIdx.x] = cap_eff[threadIdx.x];
      offv[threadIdx.x] = offsets[threadIdx.x];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 4 * kMaxE; i += 256) (&wcnt[0][0])[i] = 0;
  __syncthreads();
  const int64_t n = static_cast<int64_t>(T) * k;
  const int64_t q0 = static_cast<int64_t>(blockIdx.x) * kChunk;
  const int64_t q1 = min(n, q0 + kChunk);
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int64_t qb = q0; qb < q1; qb += 256) {
    const int64_t q = qb + threadIdx.x;
    int e = -1, t = 0, j = 0;
    if (q < q1) {
      j = static_cast<int>(q / T);
      t = static_cast<int>(q - static_cast<int64_t>(j) * T);
      if (live_assignment(ids, t, j, k, E, nullptr)) e = ids[static_cast<size_t>(t) * k + j];
    }
    const bool live = e >= 0;
    uint64_t eq = __ballot(live);
#pragma unroll
    for (int b = 0; b < 6; ++b) {
      const bool bit = live && ((e >> b) & 1);
      const uint64_t m = __ballot(bit);
      eq &= bit ? m : ~m;
    }
    int rank = 0;
    if (live) {
      rank = __popcll(eq & lt_mask);
      if (rank == 0) wcnt[wave][e] = __popcll(eq);
    }
    __syncthreads();
    if (live) {
      int pos = run[e] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][e];
      const size_t a = static_cast<size_t>(t) * k + j;
      if (pos < capv[e]) {
        const int r = offv[e] + pos;
        dest_row[a] = r;
        src[r] = static_cast<int32_t>(a);
      } else {
        dest_row[a] = -1;
      }
    } else if (q < q1) {
      dest_row[static_cast<size_t>(t) * k + j] = -1;
    }
    __syncthreads();
    if (threadIdx.x < E) {
      run[threadIdx.x] += wcnt[0][threadIdx.x] + wcnt[1][threadIdx.x] +
                          wcnt[2][threadIdx.x] + wcnt[3][threadIdx.x];
      wcnt[0][threadIdx.x] = wcnt[1][threadIdx.x] = 0;
      wcnt[2][threadIdx.x] = wcnt[3][threadIdx.x] = 0;
    }
    __syncthreads();
  }
}

// Token-major row kernels: one wavefront per token, `nvec` 16-byte vectors
// per row (row bytes / 16), lanes stride over the row. The token index and
// its picks are wave-uniform (scalar registers, scalar branches); each lane
// loads a batch of its vectors before it uses any of them (one memory
// latency per batch instead of one per 1 KB of the row), the ragged end of a
// row in smaller batches.
constexpr int kRowWaves = 4;
constexpr int kRowBatch = 4;

__device__ __forceinline__ int row_token() {
  return __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x) * kRowWaves +
                                        (static_cast<int>(threadIdx.x) >> 6));
}

// Makes a loaded value opaque to the optimiser, so that the copies below
// store the registers the batch loaded rather than loading them again per
// kept pick.
__device__ __forceinline__ void hold(uint4& v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  u32x4 r = __builtin_bit_cast(u32x4, v);
  asm volatile("" : "+v"(r));
  v = __builtin_bit_cast(uint4, r);
}

// Walks a lane's vectors v = lane, lane+64, ... < nvec in batches: f(NB, v)
// takes vectors v, v+64, ..., v+64*(NB-1), all in range. Batches of UB while
// they fit, then one of 2 (UB > 2), then single vectors.
template <int UB, typename F>
__device__ __forceinline__ void for_row_batches(int nvec, int lane, F&& f) {
  int v = lane;
  for (; v + 64 * (UB - 1) < nvec; v += 64 * UB) f(std::integral_constant<int, UB>{}, v);
  if constexpr (UB > 2) {
    if (v + 64 < nvec) {
      f(std::integral_constant<int, 2>{}, v);
      v += 128;
    }
  }
  for (; v < nvec; v += 64) f(std::integral_constant<int, 1>{}, v);
}

template <int NB>
__device__ __forceinline__ void gather_vecs(const uint4* __restrict__ xr, const int (&dst)[kMaxK],
                                            int nvec, int v, uint4* __restrict__ x_disp) {
  uint4 val[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) val[u] = xr[v + 64 * u];
#pragma unroll
  for (int u = 0; u < NB; ++u) hold(val[u]);
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (dst[j] >= 0) {
      uint4* o = x_disp + static_cast<size_t>(dst[j]) * nvec + v;
#pragma unroll
      for (int u = 0; u < NB; ++u) o[64 * u] = val[u];
    }
  }
}

// Dispatch step 4: x_disp[dest_row[t,j]] = x[t] for every kept j.
__global__ __launch_bounds__(256) void gather_rows_kernel(
    const uint4* __restrict__ x, const int32_t* __restrict__ dest_row, int T, int k,
    int nvec, uint4* __restrict__ x_disp) {
  const int t = row_token();
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  int dst[kMaxK];
  bool any = false;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    dst[j] = __builtin_amdgcn_readfirstlane(j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1);
    any |= dst[j] >= 0;
  }
  if (!any) return;
  const uint4* xr = x + static_cast<size_t>(t) * nvec;
  for_row_batches<kRowBatch>(nvec, lane, [&](auto nb, int v) {
    gather_vecs<decltype(nb)::value>(xr, dst, nvec, v, x_disp);
  });
}

// dx is the layer's last output of a step and is not read again by the
// library: it is stored non-temporally, so its lines do not stay dirty in
// the caches, to be written back while the next kernels stream their inputs.
__device__ __forceinline__ void store_stream(uint4* p, const uint4& v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
}

// Batch of the combine below: NB vectors of the row (v, v+64, ...), all
// kept rows' loads issued first, each output element summed in order j;
// STREAM stores the result non-temporally.
template <typename T, int KT, int NB, bool STREAM = false>
__device__ __forceinline__ void combine_vecs(const uint4* __restrict__ yd, const int (&dst)[KT],
                                             const float (&w)[KT], int nvec, int v,
                                             uint4* __restrict__ yr) {
  constexpr int V = Elem<T>::kVec;
  uint4 raw[NB][KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    if (dst[j] >= 0) {
      const uint4* src = yd + static_cast<size_t>(dst[j]) * nvec + v;
#pragma unroll
      for (int u = 0; u < NB; ++u) raw[u][j] = src[64 * u];
    }
  }
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      if (dst[j] >= 0) {
        float f[V];
        Elem<T>::load(raw[u][j], f);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = fmaf(w[j], f[i], acc[i]);
      }
    }
    if (STREAM)
      store_stream(yr + v + 64 * u, Elem<T>::store(acc));
    else
      yr[v + 64 * u] = Elem<T>::store(acc);
  }
}

// y[t] = sum_j kept w[t,j] * y_disp[dest_row[t,j]]  (fp32 sum in order j);
// KT >= k bounds the picks held in registers, and the batch shrinks as KT
// grows (KT rows' vectors per batch element).
template <typename T, int KT>
__global__ __launch_bounds__(256) void combine_kernel(
    const uint4* __restrict__ yd, const int32_t* __restrict__ dest_row,
    const float* __restrict__ wts, int Ttok, int k, int nvec, int64_t rows_alloc,
    uint4* __restrict__ y) {
  const int t = row_token();
  const int lane = threadIdx.x & 63;
  if (t >= Ttok) return;
  int dst[KT];
  float w[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    int r = j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1;
    if (r >= rows_alloc) r = -1;  // not a row of y_disp: treated as dropped
    dst[j] = __builtin_amdgcn_readfirstlane(r);
    w[j] = j < k ? wts[static_cast<size_t>(t) * k + j] : 0.f;
  }
  uint4* yr = y + static_cast<size_t>(t) * nvec;
  constexpr int UB = KT <= 2 ? kRowBatch : (KT <= 4 ? 2 : 1);
  for_row_batches<UB>(nvec, lane, [&](auto nb, int v) {
    combine_vecs<T, KT, decltype(nb)::value>(yd, dst, w, nvec, v, yr);
  });
}

// Batch of the combine backward below: NB vectors of dy[t] and of each kept
// row of y_disp, loads first; dot[j] accumulates in the lane's vector order.
template <typename T, int KT, int NB>
__device__ __forceinline__ void combine_bwd_vecs(const uint4* __restrict__ dr,
                                                 const uint4* __restrict__ yd,
                                                 const int (&dst)[KT], const float (&w)[KT],
                                                 float (&dot)[KT], int nvec, int v,
                                                 uint4* __restrict__ dyd) {
  constexpr int V = Elem<T>::kVec;
  uint4 rg[NB], ry[NB][KT];
#pragma unroll
  for (int u = 0; u < NB; ++u) rg[u] = dr[v + 64 * u];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    if (dst[j] >= 0) {
      const uint4* src = yd + static_cast<size_t>(dst[j]) * nvec + v;
#pragma unroll
      for (int u = 0; u < NB; ++u) ry[u][j] = src[64 * u];
    }
  }
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    float g[V];
    Elem<T>::load(rg[u], g);
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      if (dst[j] >= 0) {
        float f[V], o[V];
        Elem<T>::load(ry[u][j], f);
#pragma unroll
        for (int i = 0; i < V; ++i) {
          dot[j] = fmaf(g[i], f[i], dot[j]);
          o[i] = w[j] * g[i];
        }
        dyd[static_cast<size_t>(dst[j]) * nvec + v + 64 * u] = Elem<T>::store(o);
      }
    }
  }
}

// dweights[t,j] = <dy[t], y_disp[r]>; dy_disp[r] = w[t,j] * dy[t]
template <typename T, int KT>
__global__ __launch_bounds__(256) void combine_bwd_kernel(
    const uint4* __restrict__ dy, const uint4* __restrict__ yd,
    const int32_t* __restrict__ dest_row, const float* __restrict__ wts, int Ttok, int k,
    int nvec, int64_t rows_alloc, uint4* __restrict__ dyd, float* __restrict__ dweights) {
  const int t = row_token();
  const int lane = threadIdx.x & 63;
  if (t >= Ttok) return;
  int dst[KT];
  float w[KT], dot[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    int r = j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1;
    if (r >= rows_alloc) r = -1;  // not a row of the grouped buffers
    dst[j] = __builtin_amdgcn_readfirstlane(r);
    w[j] = j < k ? wts[static_cast<size_t>(t) * k + j] : 0.f;
    dot[j] = 0.f;
  }
  const uint4* dr = dy + static_cast<size_t>(t) * nvec;
  constexpr int UB = KT <= 2 ? kRowBatch : (KT <= 4 ? 2 : 1);
  for_row_batches<UB>(nvec, lane, [&](auto nb, int v) {
    combine_bwd_vecs<T, KT, decltype(nb)::value>(dr, yd, dst, w, dot, nvec, v, dyd);
  });
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    if (j < k) {
      const float s = wave_sum(dot[j]);
      if (lane == 0) dweights[static_cast<size_t>(t) * k + j] = dst[j] >= 0 ? s : 0.f;
    }
  }
}

// dx[t] = sum_j kept dx_disp[r_j] on the cached path (no gate term): the
// combine with unit weights (fmaf(1, f, acc) rounds as acc + f does), summed
// in float32 in order j, one rounding, stored non-temporally.
template <typename T, int KT>
__global__ __launch_bounds__(256) void row_sum_kernel(
    const uint4* __restrict__ dxd, const int32_t* __restrict__ dest_row, int Ttok, int k,
    int nvec, int64_t rows_alloc, uint4* __restrict__ dx) {
  const int t = row_token();
  const int lane = threadIdx.x & 63;
  if (t >= Ttok) return;
  int dst[KT];
  float w[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    int r = j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1;
    if (r >= rows_alloc) r = -1;
    dst[j] = __builtin_amdgcn_readfirstlane(r);
    w[j] = 1.f;
  }
  uint4* o = dx + static_cast<size_t>(t) * nvec;
  constexpr int UB = KT <= 2 ? kRowBatch : (KT <= 4 ? 2 : 1);
  for_row_batches<UB>(nvec, lane, [&](auto nb, int v) {
    combine_vecs<T, KT, decltype(nb)::value, true>(dxd, dst, w, nvec, v, o);
  });
}

// dx[t] = sum_j kept dx_disp[r_j] + dl[t] . w_g.  A wavefront takes a group
// of TG tokens (k <= KT) and one 64-vector column chunk of their rows
// (blockIdx.y), so each w_g vector is loaded once per group rather than once
// per token, and issues all of the group's row gathers at once.
template <int KT> struct DispatchBwdShape {
  static constexpr int TG = KT <= 2 ? 8 : 16 / KT;   // tokens per wavefront
};

template <typename T, int KT>
__global__ __launch_bounds__(256) void dispatch_bwd_kernel(
    const uint4* __restrict__ dxd, const int32_t* __restrict__ dest_row,
    const float* __restrict__ dl, const uint4* __restrict__ wg, int Ttok, int E, int k,
    int nvec, int64_t rows_alloc, uint4* __restrict__ dx) {
  constexpr int V = Elem<T>::kVec;
  constexpr int kTokGroup = DispatchBwdShape<KT>::TG;
  constexpr int kMaxK = KT;
  // wave-uniform token group: its routing values and dlogits come in through
  // scalar loads, read once per group rather than once per row vector
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int tg = (static_cast<int>(blockIdx.x) * kRowWaves + wave) * kTokGroup;
  const int lane = threadIdx.x & 63;
  if (tg >= Ttok) return;
  int rows[kTokGroup][kMaxK];
#pragma unroll
  for (int u = 0; u < kTokGroup; ++u)
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      int r = -1;
      if (j < k && tg + u < Ttok) r = dest_row[static_cast<size_t>(tg + u) * k + j];
      rows[u][j] = r >= 0 && r < rows_alloc ? r : -1;
    }
  const int v = static_cast<int>(blockIdx.y) * 64 + lane;
  if (v >= nvec) return;
  {
    float acc[kTokGroup][V];
    // issue every gather of the group before summing
    uint4 raw[kTokGroup][kMaxK];
#pragma unroll
    for (int u = 0; u < kTokGroup; ++u)
#pragma unroll
      for (int j = 0; j < kMaxK; ++j)
        if (j < k && rows[u][j] >= 0) raw[u][j] = dxd[static_cast<size_t>(rows[u][j]) * nvec + v];
#pragma unroll
    for (int u = 0; u < kTokGroup; ++u) {
#pragma unroll
      for (int i = 0; i < V; ++i) acc[u][i] = 0.f;
#pragma unroll
      for (int j = 0; j < kMaxK; ++j)
        if (j < k && rows[u][j] >= 0) {
          float f[V];
          Elem<T>::load(raw[u][j], f);
#pragma unroll
          for (int i = 0; i < V; ++i) acc[u][i] += f[i];
        }
    }
    {
      // four w_g vectors in flight per step
      constexpr int kEu = 4;
      for (int e0 = 0; e0 < E; e0 += kEu) {
        uint4 gv[kEu];
#pragma unroll
        for (int q = 0; q < kEu; ++q)
          if (e0 + q < E) gv[q] = wg[static_cast<size_t>(e0 + q) * nvec + v];
#pragma unroll
        for (int q = 0; q < kEu; ++q) {
          if (e0 + q >= E) break;
          float f[V];
          Elem<T>::load(gv[q], f);
#pragma unroll
          for (int u = 0; u < kTokGroup; ++u) {
            const int t = tg + u;
            const float g = t < Ttok ? dl[static_cast<size_t>(t) * E + e0 + q] : 0.f;
#pragma unroll
            for (int i = 0; i < V; ++i) acc[u][i] = fmaf(g, f[i], acc[u][i]);
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kTokGroup; ++u)
      if (tg + u < Ttok) store_stream(dx + static_cast<size_t>(tg + u) * nvec + v, Elem<T>::store(acc[u]));
  }
}

// Padded static baseline: zero rows [offsets[e] + fill[e], offsets[e] + rows[e])
// of a grouped buffer, rows[e] clamped to the expert's region and to
// rows_alloc exactly as the FFN schedule clamps it.  A wavefront takes one
// row; lane e tests expert e's unfilled range and a ballot decides.
constexpr int kPadRowsPerBlock = 16;

__global__ __launch_bounds__(256) void zero_pad_rows_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ fill,
    const int32_t* __restrict__ rows, int E, int64_t rows_alloc, int nvec,
    uint4* __restrict__ buf) {
  __shared__ int64_t lo[kMaxE], hi[kMaxE];
  if (threadIdx.x < kMaxE) {
    const int e = threadIdx.x;
    int64_t a = 0, b = 0;
    if (e < E) {
      const int64_t off = offsets[e];
      int64_t m = rows[e];
      if (off < 0 || off >= rows_alloc) m = 0;
      m = min(m, static_cast<int64_t>(offsets[e + 1]) - off);
      m = min(m, rows_alloc - off);
      m = max(m, int64_t(0));
      const int64_t fl = min(max(static_cast<int64_t>(fill[e]), int64_t(0)), m);
      a = off + fl;
      b = off + m;
    }
    lo[e] = a;
    hi[e] = b;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int i = wave; i < kPadRowsPerBlock; i += kRowWaves) {
    const int64_t r = static_cast<int64_t>(blockIdx.x) * kPadRowsPerBlock + i;
    if (r >= rows_alloc) break;
    const bool mine = lane < E && r >= lo[lane] && r < hi[lane];
    if (__ballot(mine) == 0) continue;
    uint4* row = buf + static_cast<size_t>(r) * nvec;
    for (int v = lane; v < nvec; v += 64) row[v] = make_uint4(0u, 0u, 0u, 0u);
  }
}

inline int nblocks(int64_t n, int per) { return static_cast<int>((n + per - 1) / per); }

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_count(void* stream, int T, int E, int k, const int32_t* ids,
                                int32_t* counts, int32_t* status) {
  if (!shape_ok(T, E, k) || !counts || !status) return MOE_EINVAL;
  if (T > 0 && !ids) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  MOE_TIMED("count", s);
  fill_i32_kernel<<<1, 64, 0, s>>>(counts, E, 0);
  MOE_LAUNCH_CHECK();
  const int64_t n = static_cast<int64_t>(T) * k;
  if (n > 0) {
    count_kernel<<<nblocks(n, kChunk), 256, 0, s>>>(ids, T, E, k, counts, status);
    MOE_LAUNCH_CHECK();
  }
  return MOE_OK;
}

extern "C" moe_status moe_update_capacity(void* stream, int T, int k, int E,
                                          const int32_t* counts, int num, int den,
                                          int cap_min, int row_align, int32_t* capacity,
                                          int32_t* offsets) {
  if (!shape_ok(T, E, k) || num < 1 || den < 1 || cap_min < 0) return MOE_EINVAL;
  if (row_align < 1 || row_align > kMaxRowAlign) return MOE_EINVAL;
  if (!capacity || !offsets) return MOE_EINVAL;
  if (static_cast<int64_t>(T) * E + static_cast<int64_t>(row_align - 1) * E >= (int64_t(1) << 31))
    return MOE_EINVAL;
  MOE_TIMED("capacity", static_cast<hipStream_t>(stream));
  capacity_kernel<<<1, 64, 0, static_cast<hipStream_t>(stream)>>>(
      T, k, E, counts, num, den, cap_min, row_align, capacity, offsets);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

static int route_nblk(int T, int k) {
  const int64_t n = static_cast<int64_t>(T) * k;
  return n > 0 ? nblocks(n, kChunk) : 1;
}

extern "C" size_t moe_dispatch_workspace_bytes(int T, int E, int k) {
  if (!shape_ok(T, E, k)) return 0;
  const size_t nblk = route_nblk(T, k);
  return align_up((2 * nblk * E + E) * sizeof(int32_t), 256);
}

static moe_status dispatch_args_ok(moe_dtype dt, int T, int d, int E, int k, const void* x,
                                   const int32_t* ids, const int32_t* capacity,
                                   const int32_t* offsets, int64_t rows_alloc,
                                   const int32_t* counts, const int32_t* fill,
                                   const int32_t* dest_row, const int32_t* src,
                                   const void* x_disp, const int32_t* status) {
  if (!dtype_ok(dt) || !shape_ok(T, E, k) || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (!capacity || !offsets || !counts || !fill || !status) return MOE_EINVAL;
  if (rows_alloc > 0 && (!src || !x_disp)) return MOE_EINVAL;
  if (T > 0 && (!x || !ids || !dest_row)) return MOE_EINVAL;
  if ((x && !aligned16(x)) || (x_disp && !aligned16(x_disp))) return MOE_EINVAL;
  return MOE_OK;
}

// The launches of moe_dispatch; `workspace` holds moe_dispatch_workspace_bytes.
static moe_status dispatch_launch(hipStream_t s, moe_dtype dt, int T, int d, int E, int k,
                                  const void* x, const int32_t* ids, const int32_t* capacity,
                                  const int32_t* offsets, int64_t rows_alloc, int32_t* counts,
                                  int32_t* fill, int32_t* dest_row, int32_t* src, void* x_disp,
                                  int32_t* status, void* workspace);

extern "C" moe_status moe_dispatch(void* stream, moe_dtype dt, int T, int d, int E, int k,
                                   const void* x, const int32_t* ids,
                                   const int32_t* capacity, const int32_t* offsets,
                                   int64_t rows_alloc, int32_t* counts, int32_t* fill,
                                   int32_t* dest_row, int32_t* src, void* x_disp,
                                   int32_t* status, void* workspace, size_t workspace_bytes) {
  const moe_status st = dispatch_args_ok(dt, T, d, E, k, x, ids, capacity, offsets, rows_alloc,
                                         counts, fill, dest_row, src, x_disp, status);
  if (st != MOE_OK) return st;
  const size_t need = moe_dispatch_workspace_bytes(T, E, k);
  if (!workspace || workspace_bytes < need) return MOE_EWORKSPACE;
  return dispatch_launch(static_cast<hipStream_t>(stream), dt, T, d, E, k, x, ids, capacity,
                         offsets, rows_alloc, counts, fill, dest_row, src, x_disp, status,
                         workspace);
}

static moe_status dispatch_launch(hipStream_t s, moe_dtype dt, int T, int d, int E, int k,
                                  const void* x, const int32_t* ids, const int32_t* capacity,
                                  const int32_t* offsets, int64_t rows_alloc, int32_t* counts,
                                  int32_t* fill, int32_t* dest_row, int32_t* src, void* x_disp,
                                  int32_t* status, void* workspace) {
  const int nblk = route_nblk(T, k);
  int32_t* hist = static_cast<int32_t*>(workspace);
  int32_t* base = hist + static_cast<size_t>(nblk) * E;
  int32_t* cap_eff = base + static_cast<size_t>(nblk) * E;
  {
    MOE_TIMED("route_hist", s);
    route_hist_kernel<<<nblk, 256, 0, s>>>(ids, T, E, k, nblk, rows_alloc, hist, src, status);
    MOE_LAUNCH_CHECK();
  }
  if (nblk <= kScanChunks) {
    // the rank kernel does the scan too (and writes counts and fill)
    MOE_TIMED("route_rank", s);
    route_rank_kernel<true><<<nblk, 256, 0, s>>>(ids, T, E, k, nullptr, nullptr, offsets,
                                                 dest_row, src, hist, nblk, capacity,
                                                 rows_alloc, counts, fill, status);
    MOE_LAUNCH_CHECK();
  } else {
    {
      MOE_TIMED("route_scan", s);
      route_scan_kernel<<<1, 64, 0, s>>>(hist, nblk, E, capacity, offsets, rows_alloc, base,
                                         cap_eff, counts, fill, status);
      MOE_LAUNCH_CHECK();
    }
    MOE_TIMED("route_rank", s);
    route_rank_kernel<false><<<nblk, 256, 0, s>>>(ids, T, E, k, base, cap_eff, offsets,
                                                  dest_row, src, nullptr, nblk, nullptr,
                                                  rows_alloc, nullptr, nullptr, nullptr);
    MOE_LAUNCH_CHECK();
  }
  if (T == 0) return MOE_OK;
  MOE_TIMED("dispatch_gather", s);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  gather_rows_kernel<<<nblocks(T, kRowWaves), 256, 0, s>>>(
      static_cast<const uint4*>(x), dest_row, T, k, nvec, static_cast<uint4*>(x_disp));
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

// ---- allocation-free dispatch ------------------------------------------------
// moe_dispatch_noalloc keeps the routing histograms in `scratch`, a fixed
// device array of this library, instead of a caller workspace.  Each GPU
// holds its own copy at its own address; the host looks that address up once
// per device and passes it to the kernels (the array's name in host code is
// only a host-side stand-in).  Every call on one GPU shares the array, so
// calls that overlap on one GPU race.  Nothing in it needs clearing: the
// histogram kernel writes every entry the scan and rank kernels read.
constexpr int64_t kNoAllocMaxAssignments = int64_t(1) << 21;  // T*k limit
constexpr size_t kNoAllocScratchBytes =
    (2 * static_cast<size_t>(kNoAllocMaxAssignments / kChunk) * kMaxE + kMaxE) * sizeof(int32_t);
static_assert(kNoAllocScratchBytes % 256 == 0, "scratch size is whole 256-byte blocks");

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_dev[kMaxDevices];  // device address of `scratch`, per device

// Device address of this device's `scratch` (looked up on the first call
// made with that device current).
static moe_status scratch_address(hipStream_t s, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MOE_EHIP;
  if (s != nullptr) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess) return MOE_EHIP;
    if (sdev != dev) return MOE_EINVAL;  // the stream must belong to the current device
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return MOE_EHIP;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return MOE_OK;
}

extern "C" size_t moe_dispatch_noalloc_max_assignments(void) {
  return static_cast<size_t>(kNoAllocMaxAssignments);
}

extern "C" moe_status moe_dispatch_noalloc(void* stream, moe_dtype dt, int T, int d, int E,
                                           int k, const void* x, const int32_t* ids,
                                           const int32_t* capacity, const int32_t* offsets,
                                           int64_t rows_alloc, int32_t* counts, int32_t* fill,
                                           int32_t* dest_row, int32_t* src, void* x_disp,
                                           int32_t* status) {
  const moe_status st = dispatch_args_ok(dt, T, d, E, k, x, ids, capacity, offsets, rows_alloc,
                                         counts, fill, dest_row, src, x_disp, status);
  if (st != MOE_OK) return st;
  if (static_cast<int64_t>(T) * k > kNoAllocMaxAssignments ||
      moe_dispatch_workspace_bytes(T, E, k) > kNoAllocScratchBytes)
    return MOE_EWORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  const moe_status sa = scratch_address(s, &ws);
  if (sa != MOE_OK) return sa;
  return dispatch_launch(s, dt, T, d, E, k, x, ids, capacity, offsets, rows_alloc, counts, fill,
                         dest_row, src, x_disp, status, ws);
}

// Calls f with std::integral_constant<int, KT> for the smallest pick bound
// KT in {1, 2, 4, 8} with k <= KT (templated row kernels size their per-pick
// registers by KT).
template <typename F>
static void with_pick_bound(int k, F&& f) {
  if (k <= 1) f(std::integral_constant<int, 1>{});
  else if (k <= 2) f(std::integral_constant<int, 2>{});
  else if (k <= 4) f(std::integral_constant<int, 4>{});
  else f(std::integral_constant<int, 8>{});
}

extern "C" moe_status moe_combine(void* stream, moe_dtype dt, int T, int d, int k,
                                  int64_t rows_alloc, const void* y_disp,
                                  const int32_t* dest_row, const float* weights, void* y) {
  if (!dtype_ok(dt) || T < 0 || k < 1 || k > kMaxK || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!y_disp || !dest_row || !weights || !y) return MOE_EINVAL;
  if (!aligned16(y_disp) || !aligned16(y)) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  MOE_TIMED("combine", s);
  with_pick_bound(k, [&](auto kt_tag) {
    constexpr int KT = decltype(kt_tag)::value;
    if (dt == MOE_BF16)
      combine_kernel<uint16_t, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(
          static_cast<const uint4*>(y_disp), dest_row, weights, T, k, nvec, rows_alloc,
          static_cast<uint4*>(y));
    else
      combine_kernel<float, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(
          static_cast<const uint4*>(y_disp), dest_row, weights, T, k, nvec, rows_alloc,
          static_cast<uint4*>(y));
  });
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" moe_status moe_combine_bwd(void* stream, moe_dtype dt, int T, int d, int k,
                                      int64_t rows_alloc, const void* dy, const void* y_disp,
                                      const int32_t* dest_row, const float* weights,
                                      void* dy_disp, float* dweights) {
  if (!dtype_ok(dt) || T < 0 || k < 1 || k > kMaxK || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!dy || !y_disp || !dest_row || !weights || !dy_disp || !dweights) return MOE_EINVAL;
  if (!aligned16(dy) || !aligned16(y_disp) || !aligned16(dy_disp)) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  MOE_TIMED("combine_bwd", s);
  with_pick_bound(k, [&](auto kt_tag) {
    constexpr int KT = decltype(kt_tag)::value;
    if (dt == MOE_BF16)
      combine_bwd_kernel<uint16_t, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(
          static_cast<const uint4*>(dy), static_cast<const uint4*>(y_disp), dest_row, weights,
          T, k, nvec, rows_alloc, static_cast<uint4*>(dy_disp), dweights);
    else
      combine_bwd_kernel<float, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(
          static_cast<const uint4*>(dy), static_cast<const uint4*>(y_disp), dest_row, weights,
          T, k, nvec, rows_alloc, static_cast<uint4*>(dy_disp), dweights);
  });
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" moe_status moe_dispatch_bwd(void* stream, moe_dtype dt, int T, int d, int E, int k,
                                       int64_t rows_alloc, const void* dx_disp,
                                       const int32_t* dest_row, const float* dlogits,
                                       const void* w_g, void* dx) {
  if (!dtype_ok(dt) || !shape_ok(T, E, k) || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!dx_disp || !dest_row || !dx) return MOE_EINVAL;
  if ((dlogits == nullptr) != (w_g == nullptr)) return MOE_EINVAL;
  if (!aligned16(dx_disp) || !aligned16(dx) || (w_g && !aligned16(w_g))) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  const uint4* a = static_cast<const uint4*>(dx_disp);
  const uint4* g = static_cast<const uint4*>(w_g);
  uint4* o = static_cast<uint4*>(dx);
  MOE_TIMED("dispatch_bwd", s);
  if (!dlogits) {
    with_pick_bound(k, [&](auto kt_tag) {
      constexpr int KT = decltype(kt_tag)::value;
      if (dt == MOE_BF16)
        row_sum_kernel<uint16_t, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(a, dest_row, T, k,
                                                                          nvec, rows_alloc, o);
      else
        row_sum_kernel<float, KT><<<nblocks(T, kRowWaves), 256, 0, s>>>(a, dest_row, T, k,
                                                                       nvec, rows_alloc, o);
    });
    MOE_LAUNCH_CHECK();
    return MOE_OK;
  }
  auto go = [&](auto kt_tag) {
    constexpr int KT = decltype(kt_tag)::value;
    const dim3 grid(nblocks(T, kRowWaves * DispatchBwdShape<KT>::TG), nblocks(nvec, 64));
    if (dt == MOE_BF16)
      dispatch_bwd_kernel<uint16_t, KT><<<grid, 256, 0, s>>>(a, dest_row, dlogits, g, T, E, k, nvec, rows_alloc, o);
    else
      dispatch_bwd_kernel<float, KT><<<grid, 256, 0, s>>>(a, dest_row, dlogits, g, T, E, k, nvec, rows_alloc, o);
  };
  with_pick_bound(k, go);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" moe_status moe_zero_pad_rows(void* stream, moe_dtype dt, int E, int d,
                                        const int32_t* offsets, const int32_t* fill,
                                        const int32_t* rows, int64_t rows_alloc, void* buf) {
  if (!dtype_ok(dt) || E < 1 || E > kMaxE || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (rows_alloc == 0) return MOE_OK;
  if (!offsets || !fill || !rows || !buf || !aligned16(buf)) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  MOE_TIMED("zero_pad_rows", s);
  zero_pad_rows_kernel<<<nblocks(rows_alloc, kPadRowsPerBlock), 256, 0, s>>>(
      offsets, fill, rows, E, rows_alloc, nvec, static_cast<uint4*>(buf));
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}
