// Gate of the MoE layer: linear scores, softmax, top-k and normalised
// weights (Algorithm 1, first three steps), and their backward.
//
// bf16 forward: one wavefront scores 32 tokens against up to 64 experts with
// v_mfma_f32_32x32x16_bf16 (token rows as the A operand, expert rows of w_g
// as the B operand, both K-contiguous); x is streamed from HBM exactly once
// with 64-byte contiguous runs per lane, so the kernel is HBM-bound.
// fp32 forward: one thread per token with float32 FMAs (small layers only).

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

constexpr int kGateTokPerWave = 32;
constexpr int kGateWaves = 4;

template <int NT>  // expert tiles of 32 (E <= 32*NT)
__global__ __launch_bounds__(256) void gate_fwd_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wg,
    const float* __restrict__ bias, int T, int d, int E, int k, int renorm,
    float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ weights) {
  __shared__ float sl[kGateWaves][kGateTokPerWave][65];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane & 31, half = lane >> 5;
  const int t0 = (blockIdx.x * kGateWaves + wave) * kGateTokPerWave;
  int trow = t0 + r;
  if (trow >= T) trow = T - 1;  // clamp loads; results of such rows are not stored
  const uint16_t* xr = x + static_cast<size_t>(trow) * d;
  const uint16_t* wr[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    int n = nt * 32 + r;
    wr[nt] = wg + static_cast<size_t>(n < E ? n : 0) * d;
  }
  floatx16 acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    for (int i = 0; i < 16; ++i) acc[nt][i] = 0.f;

  // K mapping shared by both operands: lane half h, MFMA i, element q
  // carries k = kb + 32h + 8i + q.
  for (int kb = 0; kb < d; kb += 64) {
    uint4 av[4];
    uint4 bv[NT][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int kk = kb + half * 32 + i * 8;
      const bool ok = kk < d;
      av[i] = ok ? *reinterpret_cast<const uint4*>(xr + kk) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const bool okb = ok && (nt * 32 + r) < E;
        bv[nt][i] = okb ? *reinterpret_cast<const uint4*>(wr[nt] + kk) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      bf16x8 a = __builtin_bit_cast(bf16x8, av[i]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        bf16x8 b = __builtin_bit_cast(bf16x8, bv[nt][i]);
        acc[nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[nt], 0, 0, 0);
      }
    }
  }
  // accumulator layout: register q holds row (q/4)*8 + 4*half + q%4, column r
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = nt * 32 + r;
    if (n < E) {
      const float b = bias ? bias[n] : 0.f;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = (q >> 2) * 8 + half * 4 + (q & 3);
        sl[wave][row][n] = acc[nt][q] + b;
      }
    }
  }
  __syncthreads();
  // logits out, coalesced along E
  for (int idx = lane; idx < kGateTokPerWave * E; idx += 64) {
    const int row = idx / E, e = idx - row * E;
    if (t0 + row < T) logits[static_cast<size_t>(t0 + row) * E + e] = sl[wave][row][e];
  }
  if (lane < kGateTokPerWave && t0 + lane < T) {
    const size_t t = t0 + lane;
    finish_token(&sl[wave][lane][0], E, k, renorm, ids + t * k, weights + t * k);
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
    const float* xr = x + static_cast<size_t>(t) * d;
    for (int e = 0; e < E; ++e) {
      const float* w = wg + static_cast<size_t>(e) * d;
      float a = 0.f;
      for (int i = 0; i < d; ++i) a = fmaf(xr[i], w[i], a);
      a += bias ? bias[e] : 0.f;
      sl[lane][e] = a;
      logits[static_cast<size_t>(t) * E + e] = a;
    }
    finish_token(&sl[lane][0], E, k, renorm, ids + static_cast<size_t>(t) * k,
                 weights + static_cast<size_t>(t) * k);
  }
}

// ---- backward ---------------------------------------------------------------
// dlogits per token (thread per token).
__global__ __launch_bounds__(64) void gate_bwd_dlogits_kernel(
    const float* __restrict__ logits, const int32_t* __restrict__ ids,
    const float* __restrict__ dweights, int T, int E, int k, int renorm,
    float* __restrict__ dlogits) {
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
    sdp[lane][e] = 0.f;
  }
  const int32_t* id = ids + static_cast<size_t>(t) * k;
  const float* dw = dweights + static_cast<size_t>(t) * k;
  float S = 0.f, dot = 0.f;
  for (int j = 0; j < k; ++j) {
    const int e = min(max(id[j], 0), E - 1);
    S += sp[lane][e];
  }
  if (renorm) {
    for (int j = 0; j < k; ++j) {
      const int e = min(max(id[j], 0), E - 1);
      dot += dw[j] * (sp[lane][e] / S);
    }
  }
  for (int j = 0; j < k; ++j) {
    const int e = min(max(id[j], 0), E - 1);
    const float g = renorm ? (dw[j] - dot) / S : dw[j];
    sdp[lane][e] += g;
  }
  float pd = 0.f;
  for (int e = 0; e < E; ++e) pd += sdp[lane][e] * sp[lane][e];
  float* out = dlogits + static_cast<size_t>(t) * E;
  for (int e = 0; e < E; ++e) out[e] = sp[lane][e] * (sdp[lane][e] - pd);
}

// dw_g partial sums: block = 64 threads x 8 columns = 512 columns, 8 experts,
// one chunk of kGbTok tokens.  grid = (E/8 groups, d/512, chunks).
constexpr int kGbTok = 256;

template <typename T>
__global__ __launch_bounds__(64) void gate_bwd_dwg_partial_kernel(
    const T* __restrict__ x, const float* __restrict__ dl, int Ttok, int d,
    int E, float* __restrict__ part) {
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
  for (int t = tb; t < te; ++t) {
    float xv[8];
    if (colok) {
      const T* xr = x + static_cast<size_t>(t) * d + c0;
      if constexpr (sizeof(T) == 2) {
        unpack8(*reinterpret_cast<const uint4*>(xr), xv);
      } else {
        const uint4 a = *reinterpret_cast<const uint4*>(xr);
        const uint4 b = *reinterpret_cast<const uint4*>(xr + 4);
        Elem<float>::load(a, xv);
        Elem<float>::load(b, xv + 4);
      }
    } else {
#pragma unroll
      for (int c = 0; c < 8; ++c) xv[c] = 0.f;
    }
    const float* dlr = dl + static_cast<size_t>(t) * E + eg;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float g = (eg + e < E) ? dlr[e] : 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[e][c] = fmaf(g, xv[c], acc[e][c]);
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

// dw_g[e,i] = sum over chunks in order
__global__ __launch_bounds__(256) void gate_bwd_dwg_reduce_kernel(
    const float* __restrict__ part, int nchunks, int n, float* __restrict__ dwg) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int c = 0; c < nchunks; ++c) s += part[static_cast<size_t>(c) * n + i];
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
  hipStream_t s = static_cast<hipStream_t>(stream);
  MOE_TIMED("gate_fwd", s);
  if (dt == MOE_BF16) {
    const int tok_per_block = kGateTokPerWave * kGateWaves;
    dim3 grid((T + tok_per_block - 1) / tok_per_block);
    if (E <= 32)
      gate_fwd_bf16_kernel<1><<<grid, 256, 0, s>>>(
          static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_g), bias,
          T, d, E, k, renorm, logits, ids, weights);
    else
      gate_fwd_bf16_kernel<2><<<grid, 256, 0, s>>>(
          static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w_g), bias,
          T, d, E, k, renorm, logits, ids, weights);
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
                                   const float* dweights, float* dlogits,
                                   float* dw_g, void* workspace,
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
    gate_bwd_dlogits_kernel<<<dim3((T + 63) / 64), 64, 0, s>>>(logits, ids, dweights, T, E,
                                                             k, renorm, dlogits);
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
