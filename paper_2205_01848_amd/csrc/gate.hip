// Gate of the MoE layer: linear scores, softmax, top-k and normalised
// weights (Algorithm 1, first three steps), and their backward.
//
// bf16 forward: one workgroup scores 32 tokens against up to 64 experts with
// v_mfma_f32_32x32x16_bf16 (token rows as the A operand, expert rows of w_g
// as the B operand, both K-contiguous), its four waves splitting K; for rows
// longer than 2048 and at most 8 experts a second kernel streams whole rows
// and forms the dot products with v_dot2.  Either way x is streamed from HBM
// exactly once, so the gate is HBM-bound.
// fp32 forward: one thread per token with float32 FMAs (small layers only).

#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "validate.hpp"

namespace moe {
namespace {

// Per-token finish: softmax, top-k with ties to the lower index, weights.
// `l` points at the token's E logits (LDS).
__device__ __forceinline__ void finish_token(const float* l, int E, int k,
                                             int renorm, int32_t* ids_out,
                                             float* w_out) {
  float m = -INFINITY;
  for (int e = 0; e < E; ++e) m = fmaxf(m, l[e]);
  float s = 0.f;
  for (int e = 0; e < E; ++e) s += expf(l[e] - m);
  uint64_t taken = 0;
  float pe[kMaxK];
  int id[kMaxK];
  float sel = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      int bi = -1;
      float best = -INFINITY;
      for (int e = 0; e < E; ++e) {
        if ((taken >> e) & 1ull) continue;
        if (bi < 0 || l[e] > best) { best = l[e]; bi = e; }
      }
      taken |= 1ull << bi;
      id[j] = bi;
      pe[j] = expf(l[bi] - m);
      sel += pe[j];
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      ids_out[j] = id[j];
      w_out[j] = renorm ? pe[j] / sel : pe[j] / s;
    }
  }
}

constexpr int kGateTile = 32;   // tokens per MFMA row tile
constexpr int kGateWaves = 4;   // waves per workgroup
constexpr int kGateStage = kGateTile * 128;   // one K step of a tile: 32 rows x 64 bf16

// Buffer resource over a whole operand; an offset of 0x80000000 is out of
// range (every real offset stays below 2^31, checked on the host), so such a
// lane reads zeros: ragged token rows, absent experts and K tails.
constexpr uint32_t kGateOob = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t gate_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           0x7FFFFFFF, 0x00020000);
}

// LDS of one wave: one K step of the tile's 32 token rows (4 KB), then the
// step's w_g rows (8 EB rows).  Row q at q * 128 bytes; its 16-byte chunk c
// at (c ^ ((q >> 1) & 7)).
template <int EB> struct GateStage {
  static constexpr int kW = kGateStage;                 // w_g rows start
  static constexpr int kBytes = kW + EB * 8 * 128;
};

// A workgroup scores kGateWaves / S token tiles of 32 tokens; the S waves of
// one tile split K: wave w of the tile takes the 64-wide K steps w, w+S, ...
// (S = 1 on long batches; 2 or 4 so that short batches still fill the chip).
// Each wave loads a K step of its tile's rows, and the step's rows of w_g,
// with 16-byte buffer loads in which 8 lanes cover one row's 128 contiguous
// bytes, so every fetched cache line is used whole by one instruction.  The
// loads run P steps ahead into a ring of registers; a step's registers go to
// the wave's LDS buffer (in-order LDS traffic within a wave needs no
// barrier), from which the MFMA operands are read.  Every step issues the
// same loads (out-of-range lanes read zeros), so the loop is branch-free and
// the compiler waits for exactly the step in use.  The S partial scores are
// summed through LDS in a fixed order.
template <int NT, int EB, int P>  // expert tiles of 32 (E <= 32*NT); w_g 8-row blocks (E <= 8*EB); steps in flight
__global__ __launch_bounds__(256) void gate_fwd_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
    const float* __restrict__ bias, int T, int d, int E, int k, int renorm,
    int S, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ weights) {
  using G = GateStage<EB>;
  constexpr int PITCH = NT * 32 + 1;  // partial-score row pitch (floats)
  constexpr int NB = 4 + EB;          // 16-byte loads per lane per K step
  static_assert(kGateTile * PITCH * 4 <= G::kBytes, "partial scores fit in a wave's buffer");
  __shared__ __attribute__((aligned(16))) char smem[kGateWaves * G::kBytes];
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int lane = threadIdx.x & 63;
  const int r = lane & 31, half = lane >> 5;
  const int tiles = kGateWaves / S;
  const int tile = wave / S, split = wave - tile * S;
  const int t0 = (blockIdx.x * tiles + tile) * kGateTile;
  const int nsteps = (d + 63) / 64;
  const int nmy = split < nsteps ? (nsteps - split + S - 1) / S : 0;   // this wave's K steps
  char* buf = smem + wave * G::kBytes;
  const __amdgpu_buffer_rsrc_t rx = gate_rsrc(x + static_cast<size_t>(t0) * d);
  const __amdgpu_buffer_rsrc_t rw = gate_rsrc(wg);
  // this lane's row within each 8-row block and its chunk, both for the
  // global read (chunk = 16 contiguous bytes) and the swizzled LDS write
  const int rowb = lane >> 3, lc = lane & 7;
  uint32_t roff[NB];      // byte offset of the lane's chunk in step 0, or out of range
  int wofs[NB];           // LDS byte offset of the lane's chunk
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) {
    const bool is_x = blk < 4;
    const int row = 8 * (is_x ? blk : blk - 4) + rowb;
    const bool ok = is_x ? t0 + row < T : row < E;
    roff[blk] = ok ? static_cast<uint32_t>(row * d * 2 + lc * 16) : kGateOob;
    wofs[blk] = (is_x ? 0 : G::kW) + row * 128 + ((lc ^ ((row >> 1) & 7)) << 4);
  }
  floatx16 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    for (int i = 0; i < 16; ++i) acc[nt][i] = 0.f;

  uint4 ring[P][NB];
  // K step j of this wave into ring slot u (zeros beyond the wave's steps
  // or beyond d)
  auto issue = [&](int j, uint4 (&slot)[NB]) {
    const int kt = split + j * S;
    // out of range as arithmetic, not a branch: setting bit 31 of an offset
    // puts it beyond the buffer (a scalar offset of 2^31 does so for steps
    // past this wave's last)
    const uint32_t kbad = static_cast<uint32_t>(kt * 64 + lc * 8 >= d) << 31;
    const int soff = j < nmy ? kt * 128 : static_cast<int>(kGateOob);
#pragma unroll
    for (int blk = 0; blk < NB; ++blk)
      slot[blk] = __builtin_bit_cast(
          uint4, __builtin_amdgcn_raw_buffer_load_b128(blk < 4 ? rx : rw, roff[blk] | kbad, soff, 0));
  };
  // issue order matters (loads complete in order): keep the compiler from
  // reordering the prologue's steps
#pragma unroll
  for (int u = 0; u < P; ++u) {
    issue(u, ring[u]);
    __builtin_amdgcn_sched_barrier(0);
  }

  // K mapping shared by both operands: step kt, MFMA i, lane half h,
  // element q carries k = 64 kt + 16 i + 8 h + q.
  const int sw = (r >> 1) & 7;
  auto step = [&](int j, uint4 (&slot)[NB]) {
#pragma unroll
    for (int blk = 0; blk < NB; ++blk) *reinterpret_cast<uint4*>(buf + wofs[blk]) = slot[blk];
    issue(j + P, slot);   // the slot's registers are in LDS: refill it
    uint4 a[4], b[NT][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = ((2 * i + half) ^ sw) << 4;
      a[i] = *reinterpret_cast<const uint4*>(buf + r * 128 + c);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        // lanes beyond the loaded w_g rows read a loaded row and use zeros
        const int n = nt * 32 + r, nr = n & (8 * EB - 1);
        const uint4 v = *reinterpret_cast<const uint4*>(
            buf + G::kW + nr * 128 + (((2 * i + half) ^ ((nr >> 1) & 7)) << 4));
        const uint32_t m = 0u - static_cast<uint32_t>(n < 8 * EB);   // all ones or zero
        b[nt][i] = make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        acc[nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[i]),
                                                          __builtin_bit_cast(bf16x8, b[nt][i]),
                                                          acc[nt], 0, 0, 0);
  };
  for (int j0 = 0; j0 < nmy; j0 += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) step(j0 + u, ring[u]);
  }

  // the buffers now hold the partial scores
  __syncthreads();
  float (*part)[PITCH] = reinterpret_cast<float (*)[PITCH]>(buf);
  // accumulator layout: register q holds row (q/4)*8 + 4*half + q%4, column r
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int row = (q >> 2) * 8 + half * 4 + (q & 3);
      part[row][nt * 32 + r] = acc[nt][q];
    }
  }
  __syncthreads();
  auto wpart = [&](int w) { return reinterpret_cast<float (*)[PITCH]>(smem + w * G::kBytes); };
  // sum each tile's K partials in split order, add the bias; logits out,
  // coalesced along E
  const int tb = blockIdx.x * tiles * kGateTile;
  for (int idx = threadIdx.x; idx < tiles * kGateTile * E; idx += 256) {
    const int row = idx / E, e = idx - row * E;
    const int tt = row / kGateTile, rr = row - tt * kGateTile;
    float v = wpart(tt * S)[rr][e];
    for (int w = 1; w < S; ++w) v += wpart(tt * S + w)[rr][e];
    v += bias ? bias[e] : 0.f;
    wpart(tt * S)[rr][e] = v;
    if (tb + row < T) logits[static_cast<size_t>(tb + row) * E + e] = v;
  }
  __syncthreads();
  const int row = threadIdx.x;
  if (row < tiles * kGateTile && tb + row < T) {
    const int tt = row / kGateTile, rr = row - tt * kGateTile;
    const size_t t = tb + row;
    finish_token(&wpart(tt * S)[rr][0], E, k, renorm, ids + t * k, weights + t * k);
  }
}

// Waves per token tile: 1 while the grid has at least 512 workgroups, else
// as many (2 or 4) as it takes to reach that or the maximum.
inline int gate_split(int T) {
  int S = 1;
  while (S < kGateWaves && (T + kGateTile * (kGateWaves / S) - 1) / (kGateTile * (kGateWaves / S)) < 512)
    S *= 2;
  return S;
}

// Whole-row bf16 gate for long rows and few experts (2048 < d <= 4096,
// E <= 8).  Read a cache line at a time from 32 rows of 8 KB at once, as
// the tiled kernel does, x streams at about 4.6 TB/s; read front to back a
// row at a time it streams at about 5.7.  Each wave scores a group of
// TPW = 4 consecutive tokens at a time, in NCH chunks of 1 KB per row: one
// 16-byte load per lane covers a contiguous kilobyte.  w_g sits in LDS
// (experts padded to 8 rows, columns to NCH chunks, both with zeros); lane
// l keeps the partial dot products of its 8 columns of every chunk for all
// 4 x 8 (token, expert) pairs, with v_dot2 (bf16 pairs, fp32 accumulation),
// and a butterfly over the lanes gives the group's 32 sums.  While a group
// is consumed chunk by chunk the same registers are refilled with the
// wave's next group, so one group (4 * NCH KB) stays in flight per wave;
// every load is issued (out-of-range lanes read zeros) and the loops have
// no branch but their own.  The logits of a batch of 32 tokens collect in
// the wave's LDS, then 32 lanes finish one token each.
// Sum of value (lane >> 1) of v[0..31] over all 64 lanes, in lanes lane and
// lane ^ 1.  Each step pairs a lane with a partner that holds the same
// subset of values, keeps one half of that subset (the upper half in the
// lane whose distinguishing bit is set) and adds the partner's copy of it:
// partners lane ^ 32 and lane ^ 16 through the permlane swaps (which move
// half of each of two registers, so no select is needed), then lane ^ 8
// (row_ror:8), 7 - lane within 8 lanes (row_half_mirror), lane ^ 2 and
// lane ^ 1 (quad_perm) through DPP.
template <int CTRL> __device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float butterfly32(const float (&v)[32], int lane) {
  float a[16], b[8], c[4], e[2];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]), __float_as_uint(v[i + 16]),
                                                    false, false);
    a[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a[i]), __float_as_uint(a[i + 8]),
                                                    false, false);
    b[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  const bool u8 = (lane & 8) != 0, u4 = (lane & 4) != 0, u2 = (lane & 2) != 0;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    c[i] = (u8 ? b[i + 4] : b[i]) + dpp<0x128>(u8 ? b[i] : b[i + 4]);
#pragma unroll
  for (int i = 0; i < 2; ++i)
    e[i] = (u4 ? c[i + 2] : c[i]) + dpp<0x141>(u4 ? c[i] : c[i + 2]);
  const float f = (u2 ? e[1] : e[0]) + dpp<0x4E>(u2 ? e[0] : e[1]);
  return f + dpp<0xB1>(f);
}

constexpr int kRowsChunk = 512;      // bf16 elements per chunk (64 lanes x 8)
constexpr int kRowsE = 8;            // experts (padded)
constexpr int kRowsTPW = 4;          // tokens per group: kRowsTPW * kRowsE = 32 values
constexpr int kRowsBatch = 32;       // tokens finished together
constexpr int kRowsMinChunks = 5;    // the tiled kernel is as fast up to d = 2048
constexpr int kRowsMaxChunks = 8;    // w_g in LDS: 8 x 8 KB

template <int NCH>
__global__ __launch_bounds__(256, 2) void gate_rows_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
    const float* __restrict__ bias, int T, int d, int E, int k, int renorm,
    float* __restrict__ logits, int32_t* __restrict__ ids, float* __restrict__ weights) {
  constexpr int EC = kRowsE, TPW = kRowsTPW;
  constexpr int FB = kRowsBatch / TPW;           // groups per batch
  constexpr int CPR = NCH * 64;                  // 16-byte chunks per LDS row
  static_assert(TPW * EC == 32, "32 values per lane");
  __shared__ uint4 wl[EC * CPR];
  __shared__ float fin[4][kRowsBatch * EC];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int ngroups = (T + TPW - 1) / TPW;
  const int gw = blockIdx.x * 4 + wave, nw = gridDim.x * 4;
  const uint32_t rowb = static_cast<uint32_t>(d) * 2;

  // w_g into LDS (rows past E and columns past d read zeros)
  {
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(wg), static_cast<short>(0), E * rowb, 0x00020000);
    constexpr int kPer = EC * CPR / 256;
    uint4 v[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = threadIdx.x + j * 256;
      const int e = i / CPR, c = i - e * CPR;
      const uint32_t off = (e * rowb + c * 16) | (static_cast<uint32_t>(c * 8 >= d) << 31);
      v[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, 0));
    }
#pragma unroll
    for (int j = 0; j < kPer; ++j) wl[threadIdx.x + j * 256] = v[j];
  }
  uint4 ring[NCH][TPW];
  // group g's chunk c into slot: bit 31 set (out of range) past the last
  // group, past T or past d, as arithmetic rather than a branch
  auto issue = [&](int g, int c, uint4 (&slot)[TPW]) {
    const __amdgpu_buffer_rsrc_t rx =
        gate_rsrc(x + static_cast<size_t>(g < ngroups ? g : 0) * TPW * d);
    const int col = c * kRowsChunk + lane * 8;
    const uint32_t cbad = static_cast<uint32_t>(col >= d) << 31;
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const uint32_t rbad = static_cast<uint32_t>(g * TPW + t >= T) << 31;   // also g >= ngroups
      const uint32_t off = (t * rowb + static_cast<uint32_t>(col) * 2) | cbad | rbad;
      slot[t] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
    }
  };
  // the wave's groups are gw, gw + nw, ...
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    issue(gw, c, ring[c]);
    __builtin_amdgcn_sched_barrier(0);
  }
  // the (token, expert) value this lane pair ends up with, and its bias
  const int idx = lane >> 1, ve = idx % EC, vt = idx / EC;
  const float lane_bias = bias != nullptr && ve < E ? bias[ve] : 0.f;
  float* my = fin[wave];
  __syncthreads();

  auto dot8 = [](const uint4& p, const uint4& q, float c) {
    c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p.x), __builtin_bit_cast(bf16x2, q.x), c, false);
    c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p.y), __builtin_bit_cast(bf16x2, q.y), c, false);
    c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p.z), __builtin_bit_cast(bf16x2, q.z), c, false);
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p.w), __builtin_bit_cast(bf16x2, q.w), c, false);
  };
  // batches of FB groups: gb, gb + nw, ..., gb + (FB - 1) * nw
  for (int gb = gw; gb < ngroups; gb += FB * nw) {
#pragma unroll 1
    for (int s = 0; s < FB && gb + s * nw < ngroups; ++s) {
      const int g = gb + s * nw;
      // w_g is read from LDS again for every group: held in registers
      // across groups it would take EC * NCH * 4 of them
      asm volatile("" ::: "memory");
      float v[32];
#pragma unroll
      for (int i = 0; i < 32; ++i) v[i] = 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const uint4* wc = wl + c * 64 + lane;
#pragma unroll
        for (int e = 0; e < EC; ++e) {
          const uint4 w = wc[e * CPR];
#pragma unroll
          for (int t = 0; t < TPW; ++t) v[t * EC + e] = dot8(ring[c][t], w, v[t * EC + e]);
        }
        issue(g + nw, c, ring[c]);   // consumed: the wave's next group
      }
      const float l = butterfly32(v, lane) + lane_bias;
      const int tok = g * TPW + vt;
      if ((lane & 1) == 0) my[s * 32 + idx] = l;
      if ((lane & 1) == 0 && ve < E && tok < T) logits[static_cast<size_t>(tok) * E + ve] = l;
    }
    // token slot lane = (group s, token t) of the batch, its logits at lane * EC
    __builtin_amdgcn_wave_barrier();
    const int tok = (gb + (lane / TPW) * nw) * TPW + lane % TPW;
    if (lane < kRowsBatch && tok < T)
      finish_token(my + lane * EC, E, k, renorm, ids + static_cast<size_t>(tok) * k,
                   weights + static_cast<size_t>(tok) * k);
    __builtin_amdgcn_wave_barrier();
  }
}

__global__ __launch_bounds__(64) void gate_fwd_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ wg,
    const float* __restrict__ bias, int T, int d, int E, int k, int renorm,
    float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ weights) {
  __shared__ float sl[64][65];
  const int lane = threadIdx.x;
  const int t = blockIdx.x * 64 + lane;
  if (t < T) {
    // the token's row is read 16 bytes at a time (d is a multiple of 8, rows
    // start 32-byte aligned), eight such loads issued before they are used,
    // and scored against 8 experts per pass: 8 independent sums, each over i
    // in order; w_g is the same for every lane
    const float* xr = x + static_cast<size_t>(t) * d;
    constexpr int kXb = 8;   // row vectors in flight
    for (int e0 = 0; e0 < E; e0 += 8) {
      float a[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) a[q] = 0.f;
      for (int i0 = 0; i0 < d; i0 += 4 * kXb) {
        float4 xv[kXb];
#pragma unroll
        for (int u = 0; u < kXb; ++u)
          if (i0 + 4 * u < d) xv[u] = *reinterpret_cast<const float4*>(xr + i0 + 4 * u);
#pragma unroll
        for (int u = 0; u < kXb; ++u) {
          const int i = i0 + 4 * u;
          if (i >= d) break;
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            if (e0 + q < E) {
              const float4 w = *reinterpret_cast<const float4*>(wg + static_cast<size_t>(e0 + q) * d + i);
              a[q] = fmaf(xv[u].x, w.x, a[q]);
              a[q] = fmaf(xv[u].y, w.y, a[q]);
              a[q] = fmaf(xv[u].z, w.z, a[q]);
              a[q] = fmaf(xv[u].w, w.w, a[q]);
            }
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int e = e0 + q;
        if (e < E) {
          const float v = a[q] + (bias ? bias[e] : 0.f);
          sl[lane][e] = v;
          logits[static_cast<size_t>(t) * E + e] = v;
        }
      }
    }
    finish_token(&sl[lane][0], E, k, renorm, ids + static_cast<size_t>(t) * k,
                 weights + static_cast<size_t>(t) * k);
  }
}

// ---- backward ---------------------------------------------------------------
// dlogits per token (thread per token).
__global__ __launch_bounds__(64) void gate_bwd_dlogits_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ ids,
    const float* __restrict__ dweights, const float* __restrict__ coef, int T, int E, int k,
    int renorm, float* __restrict__ dlogits) {
  __shared__ float sp[64][65];
  __shared__ float sdp[64][65];
  const int lane = threadIdx.x;
  const int t = blockIdx.x * 64 + lane;
  if (t >= T) return;
  const float* l = logits + static_cast<size_t>(t) * E;
  float m = -INFINITY;
  for (int e = 0; e < E; ++e) m = fmaxf(m, l[e]);
  float s = 0.f;
  for (int e = 0; e < E; ++e) {
    const float z = expf(l[e] - m);
    sp[lane][e] = z;
    s += z;
  }
  const float inv = 1.f / s;
  for (int e = 0; e < E; ++e) {
    sp[lane][e] *= inv;
    sdp[lane][e] = coef ? coef[e] : 0.f;  // a dprobs term shared by every token
  }
  const int32_t* id = ids + static_cast<size_t>(t) * k;
  const float* dw = dweights + static_cast<size_t>(t) * k;
  // An id outside [0, E) (a bad cached id) is not a pick: its weight is 0
  // and it takes no part in the normalisation, as in moe_cached_weights.
  float S = 0.f, dot = 0.f;
  for (int j = 0; j < k; ++j) {
    const int e = id[j];
    if (e >= 0 && e < E) S += sp[lane][e];
  }
  if (renorm) {
    for (int j = 0; j < k; ++j) {
      const int e = id[j];
      if (e >= 0 && e < E) dot += dw[j] * (sp[lane][e] / S);
    }
  }
  for (int j = 0; j < k; ++j) {
    const int e = id[j];
    if (e < 0 || e >= E) continue;
    const float g = renorm ? (dw[j] - dot) / S : dw[j];
    sdp[lane][e] += g;
  }
  float pd = 0.f;
  for (int e = 0; e < E; ++e) pd += sdp[lane][e] * sp[lane][e];
  float* out = dlogits + static_cast<size_t>(t) * E;
  for (int e = 0; e < E; ++e) out[e] = sp[lane][e] * (sdp[lane][e] - pd);
}

// dw_g partial sums: block = 64 threads x 8 columns = 512 columns, 8 experts,
// one chunk of kGbTok tokens.  grid = (E/8 groups, d/512, chunks).  The
// tokens of a chunk are taken kGbBatch at a time: the batch's x vectors are
// loaded before any of them is used, so the loads overlap instead of each
// waiting out its own latency.  Per column the sum runs over the tokens in
// order (batching changes only when the loads are issued).
constexpr int kGbTok = 128;
constexpr int kGbBatch = 8;

template <typename T>
__global__ __launch_bounds__(64) void gate_bwd_dwg_partial_kernel(
    const T* __restrict__ x, const float* __restrict__ dl, int Ttok, int d,
    int E, float* __restrict__ part) {
  constexpr int kVecs = sizeof(T) / 2;   // 16-byte vectors per 8 elements
  const int eg = blockIdx.x * 8;
  const int c0 = (blockIdx.y * 64 + threadIdx.x) * 8;
  const int chunk = blockIdx.z;
  const int tb = chunk * kGbTok, te = min(Ttok, tb + kGbTok);
  float acc[8][8];
#pragma unroll
  for (int e = 0; e < 8; ++e)
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[e][c] = 0.f;
  const bool colok = c0 < d;
  for (int t0 = tb; t0 < te; t0 += kGbBatch) {
    uint4 raw[kGbBatch][kVecs];
#pragma unroll
    for (int u = 0; u < kGbBatch; ++u) {
      const int t = t0 + u;
#pragma unroll
      for (int v = 0; v < kVecs; ++v) {
        raw[u][v] = (colok && t < te)
                        ? reinterpret_cast<const uint4*>(x + static_cast<size_t>(t) * d + c0)[v]
                        : make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int u = 0; u < kGbBatch; ++u) {
      const int t = t0 + u;
      if (t >= te) break;
      float xv[8];
      if constexpr (sizeof(T) == 2) {
        unpack8(raw[u][0], xv);
      } else {
        Elem<float>::load(raw[u][0], xv);
        Elem<float>::load(raw[u][kVecs - 1], xv + 4);
      }
      const float* dlr = dl + static_cast<size_t>(t) * E + eg;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float g = (eg + e < E) ? dlr[e] : 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) acc[e][c] = fmaf(g, xv[c], acc[e][c]);
      }
    }
  }
  if (!colok) return;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (eg + e >= E) break;
    float* p = part + (static_cast<size_t>(chunk) * E + eg + e) * d + c0;
    *reinterpret_cast<float4*>(p) = make_float4(acc[e][0], acc[e][1], acc[e][2], acc[e][3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(acc[e][4], acc[e][5], acc[e][6], acc[e][7]);
  }
}

// dw_g[e,i] = sum over chunks in order (loads issued 8 chunks ahead of the adds)
__global__ __launch_bounds__(256) void gate_bwd_dwg_reduce_kernel(
    const float* __restrict__ part, int nchunks, int n, float* __restrict__ dwg) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  int c = 0;
  for (; c + 8 <= nchunks; c += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = part[static_cast<size_t>(c + u) * n + i];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; c < nchunks; ++c) s += part[static_cast<size_t>(c) * n + i];
  dwg[i] = s;
}

__global__ void zero_f32_kernel(float* p, size_t n) {
  size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_gate_topk(void* stream, moe_dtype dt, int T, int d,
                                    int E, int k, int renorm, const void* x,
                                    const void* w_g, const float* bias,
                                    float* logits, int32_t* ids,
                                    float* weights) {
  if (!dtype_ok(dt) || !shape_ok(T, E, k) || !width_ok(d)) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!x || !w_g || !logits || !ids || !weights) return MOE_EINVAL;
  if (!aligned16(x) || !aligned16(w_g)) return MOE_EINVAL;
  // bf16 buffer offsets (a 32-row tile of x, all of w_g) stay below 2^31
  if (dt == MOE_BF16 && static_cast<int64_t>(d) * 2 * kMaxE >= (int64_t(1) << 31))
    return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  MOE_TIMED("gate_fwd", s);
  const int nch = (d + kRowsChunk - 1) / kRowsChunk;
  if (dt == MOE_BF16 && E <= kRowsE && nch >= kRowsMinChunks && nch <= kRowsMaxChunks) {
    // long rows, few experts: whole-row streaming, two workgroups per CU
    const int groups = (T + kRowsTPW - 1) / kRowsTPW;
    const int grid = std::min(2 * num_cus(), (groups + 3) / 4);
    auto go = [&](auto nc) {
      gate_rows_bf16_kernel<decltype(nc)::value><<<grid, 256, 0, s>>>(
          static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_g), bias, T, d, E, k,
          renorm, logits, ids, weights);
    };
    switch (nch) {
      case 5: go(std::integral_constant<int, 5>{}); break;
      case 6: go(std::integral_constant<int, 6>{}); break;
      case 7: go(std::integral_constant<int, 7>{}); break;
      default: go(std::integral_constant<int, 8>{}); break;
    }
  } else if (dt == MOE_BF16) {
    const int S = gate_split(T);
    const int tok_per_block = kGateTile * (kGateWaves / S);
    dim3 grid((T + tok_per_block - 1) / tok_per_block);
    auto go = [&](auto nt, auto eb, auto p) {
      gate_fwd_bf16_kernel<decltype(nt)::value, decltype(eb)::value, decltype(p)::value>
          <<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(x),
                                static_cast<const uint16_t*>(w_g), bias, T, d, E, k, renorm, S,
                                logits, ids, weights);
    };
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    if (E <= 8) go(I1{}, I1{}, I3{});
    else if (E <= 16) go(I1{}, I2{}, I3{});
    else if (E <= 32) go(I1{}, std::integral_constant<int, 4>{}, I3{});
    else go(I2{}, std::integral_constant<int, 8>{}, I2{});
  } else {
    gate_fwd_f32_kernel<<<dim3((T + 63) / 64), 64, 0, s>>>(
        static_cast<const float*>(x), static_cast<const float*>(w_g), bias, T, d,
        E, k, renorm, logits, ids, weights);
  }
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" size_t moe_gate_bwd_workspace_bytes(int T, int d, int E) {
  if (T < 0 || d < 1 || E < 1) return 0;
  const size_t nchunks = (static_cast<size_t>(T) + kGbTok - 1) / kGbTok;
  return align_up(nchunks * E * d * sizeof(float), 256);
}

extern "C" moe_status moe_gate_bwd(void* stream, moe_dtype dt, int T, int d,
                                   int E, int k, int renorm, const void* x,
                                   const float* logits, const int32_t* ids,
                                   const float* dweights, const float* dprob_coef,
                                   float* dlogits, float* dw_g, void* workspace,
                                   size_t workspace_bytes) {
  if (!dtype_ok(dt) || !shape_ok(T, E, k) || !width_ok(d)) return MOE_EINVAL;
  if (!dw_g) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t n = static_cast<size_t>(E) * d;
  if (T == 0) {
    MOE_TIMED("gate_bwd_zero", s);
    zero_f32_kernel<<<dim3((n + 255) / 256), 256, 0, s>>>(dw_g, n);
    MOE_LAUNCH_CHECK();
    return MOE_OK;
  }
  if (!x || !logits || !ids || !dweights || !dlogits) return MOE_EINVAL;
  if (!aligned16(x) || !aligned16(dw_g)) return MOE_EINVAL;
  const size_t need = moe_gate_bwd_workspace_bytes(T, d, E);
  if (!workspace || workspace_bytes < need) return MOE_EWORKSPACE;
  float* part = static_cast<float*>(workspace);
  const int nchunks = (T + kGbTok - 1) / kGbTok;
  {
    MOE_TIMED("gate_bwd_dlogits", s);
    gate_bwd_dlogits_kernel<<<dim3((T + 63) / 64), 64, 0, s>>>(logits, ids, dweights,
                                                             dprob_coef, T, E, k, renorm,
                                                             dlogits);
    MOE_LAUNCH_CHECK();
  }
  dim3 grid((E + 7) / 8, (d + 511) / 512, nchunks);
  {
  MOE_TIMED("gate_bwd_dwg_partial", s);
  if (dt == MOE_BF16)
    gate_bwd_dwg_partial_kernel<uint16_t><<<grid, 64, 0, s>>>(
        static_cast<const uint16_t*>(x), dlogits, T, d, E, part);
  else
    gate_bwd_dwg_partial_kernel<float><<<grid, 64, 0, s>>>(static_cast<const float*>(x),
                                                           dlogits, T, d, E, part);
  MOE_LAUNCH_CHECK();
  }
  MOE_TIMED("gate_bwd_dwg_reduce", s);
  gate_bwd_dwg_reduce_kernel<<<dim3((n + 255) / 256), 256, 0, s>>>(part, nchunks,
                                                                   static_cast<int>(n), dw_g);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}
