// Sample assignment caching (Section 4.2).
//
// The Cache operator compares the gate's fresh picks of a mini-batch with
// the picks cached for the same samples in the previous epoch, counts the
// samples whose set of experts did not change (the model metric that tells
// whether assignments have converged), and stores the fresh picks for the
// next epoch.  With caching on, the expert batches are built from the cached
// picks while the gate runs; the combine weights are then the gate's fresh
// probabilities read at the cached picks (moe_cached_weights).  The on/off
// decision with hysteresis (Section 5.3: on at >= 96% correctly cached and
// not before epoch 10, off below 90%) is a host function.

#include "common.hpp"
#include "validate.hpp"

namespace moe {
namespace {

// unchanged += number of tokens whose fresh pick set equals the cached set;
// then cache_out[t] = fresh[t] (cache_out may be `cached` itself: each thread
// reads its row before it writes it).
__global__ __launch_bounds__(256) void cache_update_kernel(const int32_t* __restrict__ fresh,
                                                           const int32_t* cached,
                                                           int32_t* cache_out, int T, int k,
                                                           int32_t* __restrict__ unchanged) {
  __shared__ int wave_count[4];
  const int t = blockIdx.x * 256 + threadIdx.x;
  bool same = false;
  if (t < T) {
    int f[kMaxK], c[kMaxK];
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      f[j] = j < k ? fresh[static_cast<size_t>(t) * k + j] : 0;
      c[j] = j < k ? cached[static_cast<size_t>(t) * k + j] : 0;
    }
    // set equality as inclusion both ways (a row may hold repeats)
    same = true;
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        bool fin = false, cin = false;
#pragma unroll
        for (int i = 0; i < kMaxK; ++i) {
          if (i < k) {
            fin |= f[j] == c[i];
            cin |= c[j] == f[i];
          }
        }
        same = same && fin && cin;
      }
    }
#pragma unroll
    for (int j = 0; j < kMaxK; ++j)
      if (j < k) cache_out[static_cast<size_t>(t) * k + j] = f[j];
  }
  const uint64_t ballot = __ballot(same);
  if ((threadIdx.x & 63) == 0) wave_count[threadIdx.x >> 6] = __popcll(ballot);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int n = wave_count[0] + wave_count[1] + wave_count[2] + wave_count[3];
    if (n) atomicAdd(unchanged, n);  // integer sum: the total does not depend on order
  }
}

// weights[t,j] = p[t, ids[t,j]] (renorm: divided by the sum over the picks)
// with p = softmax(logits[t]), evaluated exactly as the gate evaluates its
// own weights, so cached picks equal to the fresh ones give equal weights.
// An id outside [0, E) gets weight 0 and is left out of the sum.
__global__ __launch_bounds__(256) void cached_weights_kernel(const float* __restrict__ logits,
                                                             const int32_t* __restrict__ ids,
                                                             int T, int E, int k, int renorm,
                                                             float* __restrict__ weights) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  const float* l = logits + static_cast<size_t>(t) * E;
  float m = -INFINITY;
  for (int e = 0; e < E; ++e) m = fmaxf(m, l[e]);
  float s = 0.f;
  for (int e = 0; e < E; ++e) s += expf(l[e] - m);
  float pe[kMaxK];
  float sel = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    pe[j] = 0.f;
    if (j < k) {
      const int e = ids[static_cast<size_t>(t) * k + j];
      if (e >= 0 && e < E) pe[j] = expf(l[e] - m);
      sel += pe[j];
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j)
    if (j < k)
      weights[static_cast<size_t>(t) * k + j] =
          renorm ? (sel > 0.f ? pe[j] / sel : 0.f) : pe[j] / s;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_cache_update(void* stream, int T, int k, const int32_t* fresh_ids,
                                       const int32_t* cached, int32_t* cache_out,
                                       int32_t* unchanged) {
  if (T < 0 || k < 1 || k > kMaxK) return MOE_EINVAL;
  if (static_cast<int64_t>(T) * k >= (int64_t(1) << 31)) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!fresh_ids || !cached || !cache_out || !unchanged) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  MOE_TIMED("cache_update", s);
  cache_update_kernel<<<(T + 255) / 256, 256, 0, s>>>(fresh_ids, cached, cache_out, T, k,
                                                      unchanged);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" moe_status moe_cached_weights(void* stream, int T, int E, int k, int renorm,
                                         const float* logits, const int32_t* ids,
                                         float* weights) {
  if (!shape_ok(T, E, k)) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!logits || !ids || !weights) return MOE_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  MOE_TIMED("cached_weights", s);
  cached_weights_kernel<<<(T + 255) / 256, 256, 0, s>>>(logits, ids, T, E, k, renorm, weights);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

extern "C" int moe_caching_decision(int enabled, int64_t unchanged, int64_t samples, int epoch,
                                    int on_num, int on_den, int off_num, int off_den,
                                    int min_epoch) {
  if (on_den <= 0 || off_den <= 0 || on_num < 0 || off_num < 0 || unchanged < 0 ||
      samples < 0 || unchanged > samples)
    return -1;
  if (samples == 0) return enabled ? 1 : 0;
  const __int128 u = unchanged, n = samples;
  if (enabled) return u * off_den < static_cast<__int128>(off_num) * n ? 0 : 1;
  return (epoch >= min_epoch && u * on_den >= static_cast<__int128>(on_num) * n) ? 1 : 0;
}
