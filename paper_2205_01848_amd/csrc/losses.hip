// Loss-side operators of the MoE layer.
//
// Balance term (Eq. 3): B = lambda * n * sum_i T_i G_i with T_i the share of
// the batch's assignments given to expert i (counts / (T k)) and G_i the
// mean gate probability of expert i over the batch.  T_i comes from an
// arg-top-k and has no gradient, so dB/dp[t,i] = lambda n T_i / T is one
// coefficient per expert; moe_gate_bwd adds it to every token's dprobs.
//
// Specification loss (Eq. 2, with its operator appendix): AggregateSpec
// hands out the prediction of every (token, choice) pair, and the fused loss
// kernel evaluates sum_{j kept} w[t,j] * mse(target[t], O[t,j]) with both
// gradients in one pass over the rows: dL/dO goes straight into the expert
// rows (dy_disp) and dL/dw into dweights, replacing the combine backward.
//
// Reductions run in a fixed order (per-block partials, then one block), so
// every output is deterministic.

#include "common.hpp"
#include "validate.hpp"

namespace moe {
namespace {

constexpr int kBalTok = 256;  // tokens per block of the probability sums

// part[b][e] = sum over the block's tokens of softmax(logits[t])[e]: one
// thread per token, column sums by wave shuffles, then the four waves in
// order.
__global__ __launch_bounds__(256) void balance_partial_kernel(
    const float* __restrict__ logits, int T, int E, float* __restrict__ part) {
  __shared__ float wsum[4][kMaxE];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int t = blockIdx.x * kBalTok + tid;
  const float* l = logits + static_cast<size_t>(t < T ? t : 0) * E;
  float m = -INFINITY;
  for (int e = 0; e < E; ++e) m = fmaxf(m, l[e]);
  float s = 0.f;
  for (int e = 0; e < E; ++e) s += expf(l[e] - m);
  const float inv = t < T ? 1.f / s : 0.f;
  for (int e = 0; e < E; ++e) {
    const float v = wave_sum(expf(l[e] - m) * inv);
    if (lane == 0) wsum[wave][e] = v;
  }
  __syncthreads();
  if (tid < E)
    part[static_cast<size_t>(blockIdx.x) * E + tid] =
        (wsum[0][tid] + wsum[1][tid]) + (wsum[2][tid] + wsum[3][tid]);
}

// G_e = sum_b part[b][e] / T; B = lambda n sum_e T_e G_e; c_e = lambda n T_e / T.
// 256 threads: thread (g, e) sums the partials b = g, g + 4, ... of expert e.
__global__ __launch_bounds__(256) void balance_finish_kernel(
    const float* __restrict__ part, int nblk, const int32_t* __restrict__ counts, int T,
    int E, int k, float lambda, float* __restrict__ loss, float* __restrict__ coef) {
  __shared__ double acc4[4][kMaxE];
  __shared__ double term[kMaxE];
  const int e = threadIdx.x & 63, g = threadIdx.x >> 6;
  if (e < E) {
    double a = 0.0;
    for (int b = g; b < nblk; b += 4) a += part[static_cast<size_t>(b) * E + e];
    acc4[g][e] = a;
  }
  __syncthreads();
  if (g == 0 && e < E) {
    double G = (acc4[0][e] + acc4[1][e]) + (acc4[2][e] + acc4[3][e]);
    double tf = 0.0, c = 0.0;
    if (T > 0) {
      G /= T;
      tf = static_cast<double>(counts[e]) / (static_cast<double>(T) * k);
      c = static_cast<double>(lambda) * E * tf / T;
    }
    term[e] = tf * G;
    coef[e] = static_cast<float>(c);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double b = 0.0;
    for (int i = 0; i < E; ++i) b += term[i];
    *loss = static_cast<float>(static_cast<double>(lambda) * E * b);
  }
}

// AggregateSpec: out[t*k + j] = y_disp[dest_row[t,j]] if kept, else 0.
__global__ __launch_bounds__(256) void aggregate_spec_kernel(
    const uint4* __restrict__ yd, const int32_t* __restrict__ dest_row, int T, int k,
    int nvec, int64_t rows_alloc, uint4* __restrict__ out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  int dst[kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    dst[j] = j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1;
    if (dst[j] >= rows_alloc) dst[j] = -1;  // not a row of y_disp: treated as dropped
  }
  uint4* o = out + static_cast<size_t>(t) * k * nvec;
  for (int v = lane; v < nvec; v += 64) {
    uint4 val[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) val[j] = dst[j] >= 0 ? yd[static_cast<size_t>(dst[j]) * nvec + v] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) o[static_cast<size_t>(j) * nvec + v] = val[j];
  }
}

// Fused specification loss with squared error, one wavefront per token:
//   diff = O[t,j] - target[t];  L[t,j] = sum diff^2 / d
//   dy_disp[r] = w[t,j] * 2 diff / (T d);  dweights[t,j] = L[t,j] / T
//   part[block] = sum over the block's tokens of sum_j w[t,j] L[t,j]
template <typename T>
__global__ __launch_bounds__(256) void spec_loss_kernel(
    const uint4* __restrict__ yd, const int32_t* __restrict__ dest_row,
    const float* __restrict__ wts, const uint4* __restrict__ tgt, int Ttok, int k, int nvec,
    int d, int64_t rows_alloc, uint4* __restrict__ dyd, float* __restrict__ dweights,
    float* __restrict__ part) {
  constexpr int V = Elem<T>::kVec;
  __shared__ float tok_loss[4];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wave;
  const int lane = threadIdx.x & 63;
  float mine = 0.f;
  if (t < Ttok) {
    int dst[kMaxK];
    float w[kMaxK], sq[kMaxK], g[kMaxK];
    const float scale = 2.f / (static_cast<float>(Ttok) * static_cast<float>(d));
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      dst[j] = j < k ? dest_row[static_cast<size_t>(t) * k + j] : -1;
      if (dst[j] >= rows_alloc) dst[j] = -1;
      w[j] = j < k ? wts[static_cast<size_t>(t) * k + j] : 0.f;
      g[j] = w[j] * scale;
      sq[j] = 0.f;
    }
    const uint4* tr = tgt + static_cast<size_t>(t) * nvec;
    for (int v = lane; v < nvec; v += 64) {
      float y0[V];
      Elem<T>::load(tr[v], y0);
#pragma unroll
      for (int j = 0; j < kMaxK; ++j) {
        if (dst[j] >= 0) {
          float f[V], o[V];
          const size_t ro = static_cast<size_t>(dst[j]) * nvec + v;
          Elem<T>::load(yd[ro], f);
#pragma unroll
          for (int i = 0; i < V; ++i) {
            const float df = f[i] - y0[i];
            sq[j] = fmaf(df, df, sq[j]);
            o[i] = g[j] * df;
          }
          dyd[ro] = Elem<T>::store(o);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        const float L = dst[j] >= 0 ? wave_sum(sq[j]) / static_cast<float>(d) : 0.f;
        if (lane == 0) dweights[static_cast<size_t>(t) * k + j] = L / static_cast<float>(Ttok);
        mine = fmaf(w[j], L, mine);
      }
    }
  }
  if (lane == 0) tok_loss[wave] = mine;
  __syncthreads();
  if (threadIdx.x == 0)
    part[blockIdx.x] = (tok_loss[0] + tok_loss[1]) + (tok_loss[2] + tok_loss[3]);
}

// loss = (sum_b part[b]) / T, summed in a fixed order in float64
__global__ __launch_bounds__(256) void sum_partials_kernel(const float* __restrict__ part,
                                                           int n, double scale,
                                                           float* __restrict__ out) {
  __shared__ double s[256];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) acc += part[i];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (static_cast<int>(threadIdx.x) < h) s[threadIdx.x] += s[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = static_cast<float>(s[0] * scale);
}

inline int nblk(int64_t n, int per) { return static_cast<int>((n + per - 1) / per); }

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" size_t moe_balance_workspace_bytes(int T, int E) {
  if (T < 0 || E < 1 || E > kMaxE) return 0;
  return align_up(static_cast<size_t>(nblk(T, kBalTok)) * E * sizeof(float) + 4, 256);
}

extern "C" moe_status moe_balance_fwd(void* stream, int T, int E, int k, float lambda,
                                      const float* logits, const int32_t* counts,
                                      float* loss, float* dprob_coef, void* workspace,
                                      size_t workspace_bytes) {
  // lambda >= 0 and finite (NaN fails the first test)
  if (!shape_ok(T, E, k) || !(lambda >= 0.f) || !__builtin_isfinite(lambda)) return MOE_EINVAL;
  if (!counts || !loss || !dprob_coef || (T > 0 && !logits)) return MOE_EINVAL;
  const size_t need = moe_balance_workspace_bytes(T, E);
  if (!workspace || workspace_bytes < need) return MOE_EWORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* part = static_cast<float*>(workspace);
  const int nb = nblk(T, kBalTok);
  MOE_TIMED("balance_fwd", s);
  if (nb > 0) {
    balance_partial_kernel<<<nb, 256, 0, s>>>(logits, T, E, part);
    MOE_LAUNCH_CHECK();
  }
  balance_finish_kernel<<<1, 256, 0, s>>>(part, nb, counts, T, E, k, lambda, loss, dprob_coef);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" moe_status moe_aggregate_spec(void* stream, moe_dtype dt, int T, int d, int k,
                                         const void* y_disp, const int32_t* dest_row,
                                         int64_t rows_alloc, void* out) {
  if (!dtype_ok(dt) || T < 0 || k < 1 || k > kMaxK || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (static_cast<int64_t>(T) * k >= (int64_t(1) << 31)) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!dest_row || !out || (rows_alloc > 0 && !y_disp)) return MOE_EINVAL;
  if (!aligned16(out) || (y_disp && !aligned16(y_disp))) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  MOE_TIMED("aggregate_spec", s);
  aggregate_spec_kernel<<<nblk(T, 4), 256, 0, s>>>(static_cast<const uint4*>(y_disp), dest_row,
                                                   T, k, nvec, rows_alloc,
                                                   static_cast<uint4*>(out));
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" size_t moe_spec_loss_workspace_bytes(int T) {
  if (T < 0) return 0;
  return align_up(static_cast<size_t>(nblk(T, 4)) * sizeof(float) + 4, 256);
}

extern "C" moe_status moe_spec_loss(void* stream, moe_dtype dt, int T, int d, int k,
                                    const void* y_disp, const int32_t* dest_row,
                                    const float* weights, const void* target,
                                    int64_t rows_alloc, void* dy_disp, float* dweights,
                                    float* loss, void* workspace, size_t workspace_bytes) {
  if (!dtype_ok(dt) || T < 0 || k < 1 || k > kMaxK || !width_ok(d) || !rows_ok(rows_alloc))
    return MOE_EINVAL;
  if (static_cast<int64_t>(T) * k >= (int64_t(1) << 31)) return MOE_EINVAL;
  if (!loss) return MOE_EINVAL;
  const size_t need = moe_spec_loss_workspace_bytes(T);
  if (!workspace || workspace_bytes < need) return MOE_EWORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* part = static_cast<float*>(workspace);
  MOE_TIMED("spec_loss", s);
  if (T == 0) {
    sum_partials_kernel<<<1, 256, 0, s>>>(part, 0, 0.0, loss);
    MOE_LAUNCH_CHECK();
    return MOE_OK;
  }
  if (!dest_row || !weights || !target || !dweights || (rows_alloc > 0 && (!y_disp || !dy_disp)))
    return MOE_EINVAL;
  if (!aligned16(target) || (y_disp && !aligned16(y_disp)) || (dy_disp && !aligned16(dy_disp)))
    return MOE_EINVAL;
  const int nvec = static_cast<int>(static_cast<int64_t>(d) * esize(dt) / 16);
  const int nb = nblk(T, 4);
  if (dt == MOE_BF16)
    spec_loss_kernel<uint16_t><<<nb, 256, 0, s>>>(
        static_cast<const uint4*>(y_disp), dest_row, weights, static_cast<const uint4*>(target),
        T, k, nvec, d, rows_alloc, static_cast<uint4*>(dy_disp), dweights, part);
  else
    spec_loss_kernel<float><<<nb, 256, 0, s>>>(
        static_cast<const uint4*>(y_disp), dest_row, weights, static_cast<const uint4*>(target),
        T, k, nvec, d, rows_alloc, static_cast<uint4*>(dy_disp), dweights, part);
  MOE_LAUNCH_CHECK();
  sum_partials_kernel<<<1, 256, 0, s>>>(part, nb, 1.0 / T, loss);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}
