// Expert FFN of the MoE layer (the expert modules E_e of Algorithm 1) on
// dynamically sized per-expert tensors (Section 4.1), forward and backward.
//
// Every product is one persistent grouped GEMM kernel in "NT" form,
//     C[m, n] = sum_k A[m, k] * B[n, k]     (both operands K-contiguous),
// K tiles of 128 bytes, operand tiles loaded HBM -> LDS by buffer loads,
// double-buffered, with an XOR swizzle that keeps the MFMA fragment reads
// bank-conflict free.
//  * bf16 layers: 4 wavefronts on v_mfma_f32_16x16x32_bf16, two barriers
//    per K step, loads and fragment reads issued one at a time between the
//    MFMAs (ffn_gemm16_kernel), on 256x256 tiles (waves of 128x128, one
//    workgroup per CU) or, for products with few tiles per CU, 128x128
//    tiles (waves of 64x64, two workgroups per CU); both add every output's
//    products in the same order.
//  * fp32 layers: 8 wavefronts of 128x64 on v_mfma_f32_32x32x2f32 in two
//    ping-pong teams, one team's MFMAs overlapping the other's LDS reads
//    (ffn_gemm_f32_kernel); the forward of small fp32 layers instead runs
//    one wavefront per 32x32 output block (ffn_gemm_f32_tiny_kernel).
//  * var-M products (forward H, Y; backward dA, dX): the M dimension of
//    expert e is its row count, read on the device; tiles are listed by a
//    one-workgroup schedule kernel, so no host synchronisation is needed.
//  * var-K products (dW): K of expert e is its row count; the K range is
//    split into chunks only when few experts carry most rows, and split
//    partial sums are added in a fixed order (deterministic).
//  * operands whose contraction index is their row index (the weights in dA
//    and dX, both operands of dW) are read K-major through transposing LDS
//    reads; on large experts dX instead reads a transposed copy of [W1; W3]
//    that the backward writes first.
// The persistent grid maps workgroup b to XCD b % 8 and hands each XCD a
// contiguous run of tiles arranged as 4 M-tiles x 8 N-tiles, so tiles that
// share operand panels share that XCD's L2.
// Epilogues (activation, SwiGLU, activation backward, transposed stores) run
// per wavefront on its fp32 accumulators, staged 16 rows at a time through a
// private LDS strip, and write 16-byte vectors.

#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "validate.hpp"

namespace moe {
namespace {

constexpr int BM = 256;
constexpr int BN = 256;
constexpr int kThreads = 512;                     // 8 wavefronts, two per SIMD
constexpr int kRowBytes = 128;                    // one K tile of one operand row
constexpr int kTileBytes = BM * kRowBytes;        // 32 KB
constexpr int kStripRows = 16;                    // accumulator rows staged per pass
constexpr int kStripPitch = 72;                   // floats per staged row (64 + 8):
                                                  // rows 4 apart fall 32 banks apart
constexpr int kStripBytes = kStripRows * kStripPitch * 4;
constexpr int kStripsPerArray = kTileBytes / kStripBytes;
static_assert(3 * kStripsPerArray >= 16, "two staging strips per wave in three operand buffers");

constexpr int BM_S = 128;       // M tile of the two-workgroups-per-CU bf16 kernel
constexpr int kGroupM = 4;      // M tiles per scheduling group
constexpr int kXcds = 8;
constexpr int kSplitFloor = 512;  // smallest K chunk of a split dW product
constexpr int kKc = 64;           // split chunks are multiples of this many rows
constexpr int64_t kMaxOperandRowBytes = (int64_t(1) << 23) - 64;  // 256 rows < 2^31 bytes
// dx_disp up to this size is produced last in the backward (MI355X has a
// 256 MB last-level cache; measured on a 268 MB dx_disp, T = 32768 tokens of
// d = 2048, k = 2: the dispatch backward reads it in 0.077 ms instead of
// 0.126 ms; on a 1.1 GB one the dX product was 2% slower when run last)
constexpr int64_t kDxLastBytes = int64_t(512) << 20;

enum Act { ACT_RELU = 0, ACT_GELU = 1, ACT_SWIGLU = 2 };

// Device-side schedule written by schedule_kernel.
struct Sched {
  int n_mtiles;    // (expert, m0) tiles of BM rows
  int n_mtiles_s;  // (expert, m0) tiles of BM_S rows (the 128x128-tile kernel)
  int n_segs;      // (expert, k range) segments of the dW products
  int kc;          // split chunk (rows)
  int n_slots;     // partial-sum slots used
  int rows[kMaxE];    // clamped rows per expert
  int slot0[kMaxE];   // first partial slot of expert e (split experts)
  int nsplit[kMaxE];  // K segments of expert e
};

// 8 consecutive layer-dtype elements <-> 8 floats (16 bytes bf16, 32 bytes fp32)
template <typename T> __device__ __forceinline__ void store_vec(char* p, const float* v);
template <> __device__ __forceinline__ void store_vec<uint16_t>(char* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = pack8(v);
}
template <> __device__ __forceinline__ void store_vec<float>(char* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 16) = make_float4(v[4], v[5], v[6], v[7]);
}
template <typename T> __device__ __forceinline__ void load_vec(const char* p, float* v);
template <> __device__ __forceinline__ void load_vec<uint16_t>(const char* p, float* v) {
  unpack8(*reinterpret_cast<const uint4*>(p), v);
}
template <> __device__ __forceinline__ void load_vec<float>(const char* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 16);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// 8 elements as raw bits (one 16-byte vector of bf16, two of fp32), so a
// load can be issued early and decoded later.
template <typename T> struct Raw8 {
  uint4 v[sizeof(T) / 2];
  __device__ __forceinline__ void load(const char* p) {
#pragma unroll
    for (int i = 0; i < static_cast<int>(sizeof(T) / 2); ++i)
      v[i] = reinterpret_cast<const uint4*>(p)[i];
  }
  __device__ __forceinline__ void to_f(float* f) const {
    if constexpr (sizeof(T) == 2) {
      unpack8(v[0], f);
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        f[4 * i + 0] = __uint_as_float(v[i].x); f[4 * i + 1] = __uint_as_float(v[i].y);
        f[4 * i + 2] = __uint_as_float(v[i].z); f[4 * i + 3] = __uint_as_float(v[i].w);
      }
    }
  }
};

// ---------------------------------------------------------------------------
// activations (shared by forward epilogue, backward epilogue and transposes)
// ---------------------------------------------------------------------------
// The epilogues evaluate these once per output element, so they use the
// hardware base-2 exponential and reciprocal (relative error about 1e-6,
// far below the bf16 rounding of the stored results):
//   e^x = 2^(x log2 e),  sigmoid(h) = 1 / (1 + e^-h),
//   tanh(u) = 1 - 2 / (1 + e^(2u))  (both limits exact: e^(2u) -> inf or 0),
//   and GELU as h sigmoid(2u) (limits: -0 for large negative h, where the
//   exponential overflows to inf, and h for large positive h).
__device__ __forceinline__ float exp_fast(float x) {
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}
__device__ __forceinline__ float rcp_fast(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float tanh_fast(float u) {
  return 1.f - 2.f * rcp_fast(1.f + exp_fast(2.f * u));
}
__device__ __forceinline__ float act_f(float h, int act) {
  if (act == ACT_RELU) return fmaxf(h, 0.f);
  // GELU, tanh form: 0.5 h (1 + tanh(u)) = h sigmoid(2u) = h / (1 + e^(-2u)),
  // u = sqrt(2/pi) (h + 0.044715 h^3); -2u log2(e) = h (c1 + c3 h^2)
  constexpr float c1 = -2.f * 0.7978845608028654f * 1.4426950408889634f;
  constexpr float c3 = c1 * 0.044715f;
  return h * rcp_fast(1.f + __builtin_amdgcn_exp2f(h * __builtin_fmaf(c3, h * h, c1)));
}
__device__ __forceinline__ float act_grad_f(float h, int act) {
  if (act == ACT_RELU) return h > 0.f ? 1.f : 0.f;
  const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
  const float th = tanh_fast(u);
  const float du = 0.7978845608028654f * (1.f + 3.f * 0.044715f * h * h);
  return 0.5f * (1.f + th) + 0.5f * h * (1.f - th * th) * du;
}
__device__ __forceinline__ float sigm(float h) { return rcp_fast(1.f + exp_fast(-h)); }

// ---------------------------------------------------------------------------
// schedule
// ---------------------------------------------------------------------------
// Inclusive prefix sum over the 64 lanes of a wavefront.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t u = __shfl_up(v, o, 64);
    if (lane >= o) v += u;
  }
  return v;
}

// One wavefront, lane g = expert g.  Clamps every expert's rows to its region
// and to rows_alloc, and the tile count to the host bound the workspace was
// sized for, so no later kernel can index out of bounds.  The weight-gradient
// products split an expert's rows into K segments only when few experts
// carry most rows (about 512 work items over all of them).  The experts'
// tiles and segments are numbered in expert order by prefix sums; should a
// bound be exceeded (inconsistent offsets), lane 0 instead walks the experts
// in order and cuts the lists where the bounds stop them.
__global__ __launch_bounds__(64) void schedule_kernel(
    const int32_t* __restrict__ offsets, const int32_t* __restrict__ rows, int E,
    int64_t rows_alloc, int max_mtiles, int max_mtiles_s, int max_segs, int tmn_min,
    int max_slots, Sched* __restrict__ s, int2* __restrict__ mtile, int2* __restrict__ mtile_s,
    int4* __restrict__ seg) {
  const int g = threadIdx.x;
  // rows of expert g, clamped to its region and to rows_alloc
  int64_t m = 0;
  if (g < E) {
    const int64_t off = offsets[g];
    m = rows[g];
    if (off < 0 || off >= rows_alloc) m = 0;
    m = min(m, static_cast<int64_t>(offsets[g + 1]) - off);
    m = min(m, rows_alloc - off);
    m = max(m, int64_t(0));
  }
  const int64_t tiles = (m + BM - 1) / BM;
  const int64_t tiles_incl = wave_incl_scan(tiles);
  const int64_t tiles_total = __shfl(tiles_incl, 63, 64);
  const int64_t tiles_s = (m + BM_S - 1) / BM_S;
  const int64_t tiles_s_incl = wave_incl_scan(tiles_s);
  const int64_t tiles_s_total = __shfl(tiles_s_incl, 63, 64);
  const int64_t kw = (m + kKc - 1) / kKc * kKc;
  const int64_t kwork = __shfl(wave_incl_scan(kw), 63, 64);
  int64_t kc = (kwork * tmn_min + 511) / 512;
  kc = (kc + kKc - 1) / kKc * kKc;
  kc = max(kc, static_cast<int64_t>(kSplitFloor));
  const int64_t nsp = g < E ? (m > kc ? (m + kc - 1) / kc : 1) : 0;
  const int64_t segs_incl = wave_incl_scan(nsp);
  const int64_t slots_incl = wave_incl_scan(nsp > 1 ? nsp : 0);
  // totals read from lane 63 while every lane is active
  const int64_t segs_total = __shfl(segs_incl, 63, 64);
  const int64_t slots_total = __shfl(slots_incl, 63, 64);
  const bool fits = tiles_total <= max_mtiles && tiles_s_total <= max_mtiles_s &&
                    segs_total <= max_segs && slots_total <= max_slots;
  if (fits) {
    if (g < E) {
      const int mi = static_cast<int>(m);
      s->rows[g] = mi;
      const int t0 = static_cast<int>(tiles_incl - tiles);
      for (int i = 0; i < static_cast<int>(tiles); ++i) mtile[t0 + i] = make_int2(g, i * BM);
      const int t0s = static_cast<int>(tiles_s_incl - tiles_s);
      for (int i = 0; i < static_cast<int>(tiles_s); ++i) mtile_s[t0s + i] = make_int2(g, i * BM_S);
      const int n = static_cast<int>(nsp);
      const int s0 = static_cast<int>(segs_incl - nsp);
      const int q0 = static_cast<int>(slots_incl - (n > 1 ? n : 0));
      s->nsplit[g] = n;
      s->slot0[g] = n > 1 ? q0 : -1;
      for (int i = 0; i < n; ++i) {
        const int k0 = static_cast<int>(min(static_cast<int64_t>(i) * kc, m));
        const int k1 = static_cast<int>(min(static_cast<int64_t>(i + 1) * kc, m));
        seg[s0 + i] = make_int4(g, n > 1 ? k0 : 0, n > 1 ? k1 : mi, n > 1 ? q0 + i : -1);
      }
    }
    if (g == 0) {
      s->n_mtiles = static_cast<int>(tiles_total);
      s->n_mtiles_s = static_cast<int>(tiles_s_total);
      s->n_segs = static_cast<int>(segs_total);
      s->n_slots = static_cast<int>(slots_total);
      s->kc = static_cast<int>(kc);
    }
    return;
  }
  if (g != 0) return;
  int nm = 0, nms = 0;
  int64_t kwork_c = 0;
  for (int e = 0; e < E; ++e) {
    const int64_t off = offsets[e];
    int64_t me = rows[e];
    if (off < 0 || off >= rows_alloc) me = 0;
    me = min(me, static_cast<int64_t>(offsets[e + 1]) - off);
    me = min(me, rows_alloc - off);
    me = max(me, int64_t(0));
    me = min(me, static_cast<int64_t>(max_mtiles - nm) * BM);
    me = min(me, static_cast<int64_t>(max_mtiles_s - nms) * BM_S);
    const int mi = static_cast<int>(me);
    s->rows[e] = mi;
    for (int m0 = 0; m0 < mi; m0 += BM) mtile[nm++] = make_int2(e, m0);
    for (int m0 = 0; m0 < mi; m0 += BM_S) mtile_s[nms++] = make_int2(e, m0);
    kwork_c += (mi + kKc - 1) / kKc * kKc;
  }
  s->n_mtiles = nm;
  s->n_mtiles_s = nms;
  int64_t kcc = (kwork_c * tmn_min + 511) / 512;
  kcc = (kcc + kKc - 1) / kKc * kKc;
  kcc = max(kcc, static_cast<int64_t>(kSplitFloor));
  int ns = 0, slots = 0;
  for (int e = 0; e < E; ++e) {
    const int kp = s->rows[e];
    int ne = kp > kcc ? static_cast<int>((kp + kcc - 1) / kcc) : 1;
    if (ne > 1 && (slots + ne > max_slots || ns + ne > max_segs)) ne = 1;
    if (ns + ne > max_segs) ne = 0;
    s->nsplit[e] = ne;
    s->slot0[e] = ne > 1 ? slots : -1;
    for (int i = 0; i < ne; ++i) {
      const int k0 = static_cast<int>(min(static_cast<int64_t>(i) * kcc, static_cast<int64_t>(kp)));
      const int k1 = static_cast<int>(min(static_cast<int64_t>(i + 1) * kcc, static_cast<int64_t>(kp)));
      seg[ns++] = make_int4(e, ne > 1 ? k0 : 0, ne > 1 ? k1 : kp, ne > 1 ? slots + i : -1);
    }
    if (ne > 1) slots += ne;
  }
  s->n_segs = ns;
  s->n_slots = slots;
  s->kc = static_cast<int>(kcc);
}

// ---------------------------------------------------------------------------
// GEMM core
// ---------------------------------------------------------------------------
// c += a * b over four k values: one 32x32 fp32 block, k = 4 consecutive
// values per lane (one 32-bit element of each of the four words)
__device__ __forceinline__ void mma_f32(floatx16& c, const uint4& a, const uint4& b) {
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
}

// Operand layouts.  Every product is C[m, n] = sum_k A[m, k] B[n, k]; an
// operand is stored either K-contiguous (rows are m (or n), k along each
// row: activations in the forward, weights as out x in) or K-major (rows are
// k, m along each row: the weights in the data-gradient products, and both
// operands of the weight-gradient products, which contract over the
// dispatched rows).
enum Layout { L_KC = 0, L_KM = 1 };

// One operand of one tile (byte pointers, byte strides).
//  KC: base = tile row 0 at k = 0; rows = valid tile rows.
//  KM: base = k-row 0 at tile column 0; rows = valid tile columns; k-rows at
//      or past `split` come from base2 (k counted from split), else base.
//  Gated forward (KC B only): base holds the W1 rows, base2 the W3 rows.
struct Operand {
  const char* base;
  const char* base2;
  int64_t ld;         // bytes between consecutive rows
  int rows;
  int split;
};
struct TileOps {
  Operand a, b;
  int K;              // valid k values; rows / columns / k past the valid ones read as 0
};

// KC LDS tile: row r (0..255) of 128 bytes, its 16-byte chunk c stored at
// r*128 + ((c ^ ((r >> 1) & 7)) << 4).  gfx950 LDS serves 16 lanes of a
// 16-byte access per cycle from 64 banks (256 bytes): the MFMA fragment reads
// touch 16 consecutive rows at one logical chunk; rows alternate bank halves
// and (r >> 1) & 7 spreads each half's 8 rows over its 8 slots.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }
// KM LDS tile: k-row r of 256 elements, its 32-element segment g stored at
// segment g ^ (r & 3).  A transpose read takes, per 32-lane half, 4
// consecutive k-rows of one 32-element segment (64 bytes of bf16 each); the
// XOR puts those rows in 4 different quarters of the 256-byte bank space.

// Buffer resource over an operand.  Every offset used is below 2^31 (host
// limits; K-major resources are re-based every K step), so 0x80000000 is
// always out of range: a lane given that offset loads zeros, which is how
// ragged rows, columns and K tails are filled.
constexpr uint32_t kOob = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const char* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), static_cast<short>(0),
                                           0x7FFFFFFF, 0x00020000);
}
#define MOE_LDS(p) ((__attribute__((address_space(3))) void*)(p))

typedef short v4s __attribute__((ext_vector_type(4)));
// 4 bf16 of one k-row run, transposed across each 16-lane group (gfx950
// ds_read_b64_tr_b16): lane i = 4a + b of a group gets element b of the run
// addressed by lanes 4r + a, for r = 0..3.
__device__ __forceinline__ uint2 read_tr(const char* p) {
  const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)(p));
  return __builtin_bit_cast(uint2, v);
}

// fp32 layers: acc += A_tile * B_tile^T over the whole K extent with 8
// wavefronts in two teams of four, one wave of each team per SIMD.  Team t
// computes tile rows 128t..128t+127, its wave q columns 64q..64q+63 (gated
// forward: hidden units 32q..32q+31, W1 then W3).  Each half K step (16
// values) is a memory phase (12 fragments, LDS -> registers) followed by an
// MFMA phase (16 block products of four v_mfma_f32_32x32x2f32 each).  Team 1
// runs one barrier behind team 0, so while one wave of a SIMD issues MFMAs
// the other reads LDS.  Operand tiles go HBM -> LDS with buffer_load ... lds
// (no register staging), issued by team 0 one step ahead into the other of
// two stages.  FULL: every tile row and column is valid; K tails are checked
// per step either way.
template <int ALAY, int BLAY, bool GATED, bool FULL>
__device__ __forceinline__ void mainloop_f32(const TileOps& op, char* la0, char* lb0, char* la1,
                                             char* lb1, floatx16 (&acc)[4][2]) {
  constexpr int ES = 4;                   // bytes per element
  constexpr int KSTEP = kRowBytes / ES;   // k values per step (KC: 128 bytes per row)
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int team = wave >> 2, wq = wave & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  const int K = op.K;
  const int nk = (K + KSTEP - 1) / KSTEP;
  if (nk <= 0) return;
  const int nk2 = (nk + 1) & ~1;   // odd counts load one all-zero step

  // ---- loads.  A 1 KB load covers one 8-row block of a KC tile (lane l ->
  // row 8 blk + (l >> 3), physical chunk l & 7, logical chunk (l & 7) ^
  // swz(row), depending on the parity of blk only), or one k-row of a KM
  // tile (lane l -> physical elements 4l .. 4l + 3 of k-row blk, column =
  // segment swizzled by k & 3).
  const int l3 = lane >> 3;
  const int co0 = ((lane & 7) ^ swz(l3)) * 16, co1 = ((lane & 7) ^ swz(l3 + 8)) * 16;
  const int pe = lane * 4;                // KM physical element
  // KM column of the lane for k-row residue q = k & 3
  auto km_col = [&](int q) { return (((pe >> 5) ^ q) << 5) + (pe & 31); };
  auto ld_of = [&](const Operand& o) { return static_cast<int>(o.ld); };

  // one operand, one block, one K step.  rs/rs2: resources (KM: of this step)
  auto load_op = [&](auto lay, const Operand& o, const __amdgpu_buffer_rsrc_t& rs,
                     const __amdgpu_buffer_rsrc_t& rs2, char* dst, int blk, int kt, bool kfull,
                     bool kany, bool gated) {
    constexpr int LAY = decltype(lay)::value;
    uint32_t off;
    int soff;
    bool second = false;
    if constexpr (LAY == L_KC) {
      const int co = (blk & 1) ? co1 : co0;
      // gated forward: W1/W3 groups of 32 rows
      const int row0 = gated ? (blk >> 3) * 32 + (blk & 3) * 8 : blk * 8;
      second = gated && ((blk >> 2) & 1);
      off = static_cast<uint32_t>(l3 * ld_of(o)) + co;
      soff = row0 * ld_of(o) + kt * kRowBytes;
      if (!FULL || !kfull) {
        const bool ok = (FULL || row0 + l3 < o.rows) && (kfull || kt * kRowBytes + co < K * ES);
        if (!ok) off = kOob;
      }
    } else {
      const int krel = blk;                        // the block's k-row in the step
      const int kabs = kt * KSTEP + krel;
      const int q = krel & 3;                      // k & 3 (steps are multiples of 4 rows)
      const int col = km_col(q);
      second = kabs >= o.split;
      off = static_cast<uint32_t>(col * ES);
      soff = krel * ld_of(o);
      if (!FULL || !kfull) {
        const bool ok = (FULL || col < o.rows) && (kfull || kabs < K);
        if (!ok) off = kOob;
      }
    }
    if (!kany) off = kOob;
    if (second)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
  };
  using KC_ = std::integral_constant<int, L_KC>;
  using KM_ = std::integral_constant<int, L_KM>;
  // resources: KC operands over the whole tile, KM operands re-based per step
  const __amdgpu_buffer_rsrc_t ra_t = tile_rsrc(op.a.base);
  const __amdgpu_buffer_rsrc_t rb_t = tile_rsrc(op.b.base);
  const __amdgpu_buffer_rsrc_t rb3_t = tile_rsrc(GATED ? op.b.base2 : op.b.base);
  auto km_rsrc = [&](const Operand& o, int kt, bool second) {
    const int64_t k = static_cast<int64_t>(kt) * KSTEP - (second ? o.split : 0);
    return tile_rsrc((second ? o.base2 : o.base) + k * o.ld);
  };
  auto load = [&](int kt, char* sa, char* sb, int b0, int nb) {
    const bool kfull = (kt + 1) * KSTEP <= K;   // wave-uniform
    const bool kany = kt * KSTEP < K;
    __amdgpu_buffer_rsrc_t ra = ra_t, ra2 = ra_t, rb = rb_t, rb2 = rb3_t;
    if constexpr (ALAY == L_KM) {
      ra = km_rsrc(op.a, kt, false);
      ra2 = op.a.base2 ? km_rsrc(op.a, kt, true) : ra;
    }
    if constexpr (BLAY == L_KM) {
      rb = km_rsrc(op.b, kt, false);
      rb2 = op.b.base2 ? km_rsrc(op.b, kt, true) : rb;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < nb) {
        if constexpr (ALAY == L_KC) load_op(KC_{}, op.a, ra, ra2, sa, b0 + i, kt, kfull, kany, false);
        else load_op(KM_{}, op.a, ra, ra2, sa, b0 + i, kt, kfull, kany, false);
        if constexpr (BLAY == L_KC) load_op(KC_{}, op.b, rb, rb2, sb, b0 + i, kt, kfull, kany, GATED);
        else load_op(KM_{}, op.b, rb, rb2, sb, b0 + i, kt, kfull, kany, false);
      }
    }
  };

  // ---- fragments.  MFMA operand of lane l: row/column l % 32 of the
  // sub-tile, k values 4 (2s + l / 32) .. +3 of sub-step s.
  const int fr_row = lane & 31;
  // KC: 16-byte reads of row fr_row
  const int fr_a = (team * 128 + fr_row) * kRowBytes;
  const int fr_b = (wq * 64 + fr_row) * kRowBytes;
  // KM: four 4-byte reads, one per k-row (k-row c at physical segment
  // (column >> 5) ^ c, the swizzle of the loads)
  auto km_frag = [&](const char* st, int cb, int s) -> uint4 {
    const int k0 = 4 * (2 * s + (lane >> 5));
    uint32_t v[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int phys = (((cb >> 5) ^ c) << 5) + fr_row;
      v[c] = *reinterpret_cast<const uint32_t*>(st + (k0 + c) * 1024 + phys * 4);
    }
    return make_uint4(v[0], v[1], v[2], v[3]);
  };
  uint4 fa[4][2], fb[2][2];   // [sub-tile][k sub-step within the half step]
  // fragments of k sub-steps 2h and 2h+1 (one half of a K step)
  auto fread = [&](const char* sa, const char* sb, int h) {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int s = 2 * h + s2;
      const int sw = ((2 * s + (lane >> 5)) ^ swz(fr_row)) << 4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (ALAY == L_KC)
          fa[i][s2] = *reinterpret_cast<const uint4*>(sa + fr_a + i * 32 * kRowBytes + sw);
        else
          fa[i][s2] = km_frag(sa, team * 128 + i * 32, s);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (BLAY == L_KC)
          fb[j][s2] = *reinterpret_cast<const uint4*>(sb + fr_b + j * 32 * kRowBytes + sw);
        else
          fb[j][s2] = km_frag(sb, wq * 64 + j * 32, s);
      }
    }
  };
  auto mma = [&]() {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) mma_f32(acc[i][j], fa[i][s2], fb[j][s2]);
  };
  // s_waitcnt immediates (gfx9 encoding)
  constexpr int kWaitVm0 = 0x0F70;    // vmcnt(0)
  constexpr int kWaitLgkm0 = 0xC07F;  // lgkmcnt(0)
  // one ping-pong phase pair: read half h of a stage, then its 16 block products
  // A wave whose rows or columns of the tile are all beyond the valid ones
  // (the ragged last tile of an expert, the last column tile) skips its
  // reads and MFMAs; it still takes part in every barrier.  Its accumulators
  // stay zero and the epilogue stores none of them.
  bool active = true;
  if constexpr (!FULL) {
    const int wcols = GATED ? 32 : 64;   // the wave's columns (gated: hidden units)
    active = team * 128 < op.a.rows && wq * wcols < op.b.rows;
  }
  auto half = [&](const char* sa, const char* sb, int h, bool wait_loads) {
    if (active) fread(sa, sb, h);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (active) mma();
    __builtin_amdgcn_sched_barrier(0);
    if (wait_loads) __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __builtin_amdgcn_s_barrier();
  };

  load(0, la0, lb0, wave * 4, 4);    // stage 0: all eight waves
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();
  if (team == 0) {
    // team 0 also loads stage kt+1 at the start of step kt and waits for it
    // at the end of the step, four phases later
    for (int kt = 0; kt < nk2; kt += 2) {
      load(kt + 1, la1, lb1, wq * 8, 8);
      half(la0, lb0, 0, false);
      half(la0, lb0, 1, true);
      if (kt + 2 < nk2) load(kt + 2, la0, lb0, wq * 8, 8);
      half(la1, lb1, 0, false);
      half(la1, lb1, 1, true);
    }
    __builtin_amdgcn_s_barrier();
  } else {
    __builtin_amdgcn_s_barrier();
    for (int kt = 0; kt < nk2; kt += 2) {
      half(la0, lb0, 0, false);
      half(la0, lb0, 1, false);
      half(la1, lb1, 0, false);
      half(la1, lb1, 1, false);
    }
  }
  // every wave has passed the last barrier after its last LDS read: the
  // operand buffers are free
}

// Stage rows [16h, 16h+16) of the wave's accumulator row-block i (32 rows x
// 64 columns) as fp32, row pitch kStripPitch: the lane's registers q in
// [8h, 8h+8) hold those rows.
__device__ __forceinline__ void stage_strip(float* strip, const floatx16 (&acc)[4][2], int i,
                                            int h) {
  const int lane = threadIdx.x & 63;
  const int half = lane >> 5, col = lane & 31;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int q = 8 * h; q < 8 * h + 8; ++q) {
      const int row = ((q >> 2) - 2 * h) * 8 + half * 4 + (q & 3);
      strip[row * kStripPitch + j * 32 + col] = acc[i][j][q];
    }
}

// ---------------------------------------------------------------------------
// kernel parameters
// ---------------------------------------------------------------------------
enum Mode {
  M_FWD1 = 0,        // H = X W1^T -> A = act(H) [, H saved]
  M_FWD1_SWIGLU = 1, // H1, H3 -> A = silu(H1) H3 [, H1 H3 saved]
  M_STORE = 2,       // plain store (Y, dX)
  M_BWD_DA = 3,      // dA = dY W2 -> dH = dA act'(H)
  M_BWD_DA_SWIGLU = 4,
  M_DW = 5           // var-K weight gradient, fp32
};

struct GemmParams {
  // operands (bytes).  var-M: A rows of the dispatched buffer, B the
  // expert's weights (B2: W3 of the gated forward, or the k-rows from split
  // on of a K-major B).  var-K: A and B dispatched buffers read K-major.
  const char* A; int64_t lda;
  const char* B; const char* B2; int64_t ldb; int64_t b_gstride;
  int K;              // var-M: k values
  int kmsplit;        // var-M, K-major B: first k-row taken from B2
  int N;              // output columns
  int M_out;          // var-K: output rows
  int ntiles;         // tiles along N
  int mtiles_out;     // var-K: tiles along M
  int act;
  // outputs
  char* C; int64_t ldc;           // row-major output (bytes per row)
  char* H1; char* H3; int64_t ldh; // saved / read pre-activations (bytes per row)
  int f;                           // SwiGLU: width of one half
  float* dwA; float* dwB; int64_t dw_gstride; int split_row;
  float* partial; int64_t slot_elems;
  const int32_t* offsets;
  const Sched* sched;
  const int2* mtile;
  const int4* seg;
};

// tile order: groups of kGroupM M-tiles, N-major inside a group
__device__ __forceinline__ void decode_grouped(int L, int n_mt, int n_nt, int& mt, int& nt) {
  const int full = (n_mt / kGroupM) * kGroupM * n_nt;
  if (L < full) {
    const int grp = L / (kGroupM * n_nt);
    const int rem = L - grp * kGroupM * n_nt;
    nt = rem / kGroupM;
    mt = grp * kGroupM + (rem - nt * kGroupM);
  } else {
    const int rem = L - full;
    const int gm = n_mt - (n_mt / kGroupM) * kGroupM;
    nt = rem / gm;
    mt = (n_mt / kGroupM) * kGroupM + (rem - nt * gm);
  }
}

// bf16 tile order, two levels above each XCD's kGroupM x 8 block of tiles.
// Tiles come in bands of kBandM M-tiles; inside a band, in N-blocks of 8
// columns, and inside an N-block, in M-blocks of kGroupM rows whose tiles
// run M fastest.  The blocks of one N-block follow each other, so the 8
// blocks in flight at once (one per XCD) are 2 N-blocks x 4 M-blocks: 16 x
// 16 tiles that read 16 + 16 operand panels, against 4 + 64 when the XCDs
// take 8 N-blocks of the same 4 M-tiles, and a band's A panels stay in the
// last-level cache while its weight panels stream past.  Partial bands and
// blocks at the edges keep the same order with fewer rows or columns.
constexpr int kBandM = 4 * kGroupM;
__device__ __forceinline__ void decode_banded(int L, int n_mt, int n_nt, int& mt, int& nt) {
  const int full_bands = n_mt / kBandM;
  int r, m0, bh;
  if (L < full_bands * kBandM * n_nt) {
    const int band = L / (kBandM * n_nt);
    r = L - band * kBandM * n_nt;
    m0 = band * kBandM;
    bh = kBandM;
  } else {
    r = L - full_bands * kBandM * n_nt;
    m0 = full_bands * kBandM;
    bh = n_mt - m0;
  }
  const int full_nb = n_nt / 8;
  int n0, w;
  if (r < full_nb * 8 * bh) {
    const int nb = r / (8 * bh);
    r -= nb * 8 * bh;
    n0 = nb * 8;
    w = 8;
  } else {
    r -= full_nb * 8 * bh;
    n0 = full_nb * 8;
    w = n_nt - n0;
  }
  const int full_mb = bh / kGroupM;
  int h;
  if (r < full_mb * kGroupM * w) {
    const int mb = r / (kGroupM * w);
    r -= mb * kGroupM * w;
    m0 += mb * kGroupM;
    h = kGroupM;
  } else {
    r -= full_mb * kGroupM * w;
    m0 += full_mb * kGroupM;
    h = bh - full_mb * kGroupM;
  }
  mt = m0 + r % h;
  nt = n0 + r / h;
}

// The products: PASS names the instance (so each is its own kernel in
// traces) and fixes the operand layouts.
// P_BWD_DX_T is dX with the weights read from a transposed copy,
// K-contiguous like the forward's operands.
enum Pass {
  P_FWD_H = 0, P_FWD_Y = 1, P_BWD_DA = 2, P_BWD_DX = 3, P_BWD_DW2 = 4, P_BWD_DW13 = 5,
  P_BWD_DX_T = 6
};
__host__ __device__ constexpr int a_layout(int pass) {
  return pass == P_BWD_DW2 || pass == P_BWD_DW13 ? L_KM : L_KC;
}
__host__ __device__ constexpr int b_layout(int pass) {
  return pass == P_BWD_DA || pass == P_BWD_DX || pass == P_BWD_DW2 || pass == P_BWD_DW13 ? L_KM
                                                                                          : L_KC;
}

template <int MODE, int PASS>
__global__ __launch_bounds__(kThreads, 1) void ffn_gemm_f32_kernel(const GemmParams p) {
  // two stages of the A and B tiles, four distinct objects (see mainloop);
  // after the K loop the same memory holds each wave's epilogue strip
  __shared__ __attribute__((aligned(16))) char la0[kTileBytes];
  __shared__ __attribute__((aligned(16))) char lb0[kTileBytes];
  __shared__ __attribute__((aligned(16))) char la1[kTileBytes];
  __shared__ __attribute__((aligned(16))) char lb1[kTileBytes];
  using T = float;
  constexpr int ES = 4;
  constexpr bool VARK = MODE == M_DW;
  constexpr bool GATED = MODE == M_FWD1_SWIGLU;
  constexpr int ALAY = a_layout(PASS), BLAY = b_layout(PASS);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int team = wave >> 2, wq = wave & 3;
  const Sched& sc = *p.sched;
  const int n_items = VARK ? sc.n_segs * p.mtiles_out * p.ntiles : sc.n_mtiles * p.ntiles;
  const int G = gridDim.x;
  const int lbase = (blockIdx.x % kXcds) * (G / kXcds) + blockIdx.x / kXcds;
  // the wave's staging strip (kStripsPerArray per 32 KB array)
  auto strip_at = [&](int sidx) {
    const int arr = sidx / kStripsPerArray, off = (sidx % kStripsPerArray) * kStripBytes;
    char* base = arr == 0 ? la0 : (arr == 1 ? lb0 : la1);
    return reinterpret_cast<float*>(base + off);
  };

  for (int round = 0;; ++round) {
    const int L = round * G + lbase;
    if (L >= n_items) break;
    // An opaque zero, produced inside the tile loop: the per-lane epilogue
    // addresses derived from it are computed per tile instead of being
    // hoisted out of the loop and held (or spilled) across the K loop.
    int z;
    asm volatile("s_mov_b32 %0, 0" : "=s"(z));
    float* strip = strip_at(2 * wave) + z;
    TileOps op;
    int g, row0, m_valid;       // var-M: expert, first global row, valid rows in tile
    int n0;                      // first output column of the tile
    int slot = -1, mt, nt;
    if constexpr (!VARK) {
      int mti;
      decode_grouped(L, sc.n_mtiles, p.ntiles, mti, nt);
      const int2 tm = p.mtile[mti];
      g = tm.x;
      row0 = p.offsets[g] + tm.y;
      m_valid = min(BM, sc.rows[g] - tm.y);
      op.a = {p.A + static_cast<int64_t>(row0) * p.lda, nullptr, p.lda, m_valid, 0};
      op.K = p.K;
      const char* bg = p.B + static_cast<int64_t>(g) * p.b_gstride;
      if constexpr (GATED) {
        n0 = nt * (BN / 2);  // hidden units covered by this tile (W1 and W3 rows)
        op.b = {bg + static_cast<int64_t>(n0) * p.ldb,
                p.B2 + static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0) * p.ldb,
                p.ldb, min(BN / 2, p.N - n0), 0};
      } else if constexpr (BLAY == L_KC) {
        n0 = nt * BN;
        op.b = {bg + static_cast<int64_t>(n0) * p.ldb, nullptr, p.ldb, min(BN, p.N - n0), 0};
      } else {  // K-major weights: k-row 0, column n0
        n0 = nt * BN;
        op.b = {bg + static_cast<int64_t>(n0) * ES,
                p.B2 ? p.B2 + static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0) * ES
                     : nullptr,
                p.ldb, min(BN, p.N - n0), p.B2 ? p.kmsplit : 0x7FFFFFFF};
      }
    } else {
      const int tmn = p.mtiles_out * p.ntiles;
      const int si = L / tmn;
      decode_grouped(L - si * tmn, p.mtiles_out, p.ntiles, mt, nt);
      const int4 sg = p.seg[si];
      g = sg.x;
      slot = sg.w;
      // this segment's dispatched rows: offsets[g] + [k0, k1) of the expert
      const int k1 = min(sg.z, sc.rows[g]);
      const int64_t krow = static_cast<int64_t>(p.offsets[g]) + sg.y;
      row0 = mt * BM;
      n0 = nt * BN;
      m_valid = min(BM, p.M_out - row0);
      op.a = {p.A + krow * p.lda + static_cast<int64_t>(row0) * ES, nullptr, p.lda, m_valid,
              0x7FFFFFFF};
      op.b = {p.B + krow * p.ldb + static_cast<int64_t>(n0) * ES, nullptr, p.ldb,
              min(BN, p.N - n0), 0x7FFFFFFF};
      op.K = max(0, k1 - sg.y);
    }

    floatx16 acc[4][2];
    if (op.a.rows >= BM && op.b.rows >= (GATED ? BN / 2 : BN))
      mainloop_f32<ALAY, BLAY, GATED, true>(op, la0, lb0, la1, lb1, acc);
    else
      mainloop_f32<ALAY, BLAY, GATED, false>(op, la0, lb0, la1, lb1, acc);

    // Epilogue, wave by wave: 16 accumulator rows at a time go through the
    // wave's own LDS strip, then each lane finishes 8 consecutive columns of
    // a row and writes them as one vector.
    const int wcol = wq * 64;   // the wave's first tile column
    if constexpr (MODE == M_BWD_DA || MODE == M_BWD_DA_SWIGLU) {
      // dH = dA act'(H): 16 (row block, strip half, row group) iterations,
      // each reading 8 saved pre-activations (two planes for SwiGLU) per
      // lane.  Those loads run kPf iterations ahead of their use, so the
      // wave waits for HBM once per tile rather than once per iteration.
      constexpr bool SW = MODE == M_BWD_DA_SWIGLU;
      constexpr int kIt = 16, kPf = 4;
      Raw8<T> q1[kIt], q3[kIt];
      auto pos = [&](int n, int& lm, int& gc) {
        const int i = n >> 2, h = (n >> 1) & 1, it = n & 1;
        lm = team * 128 + i * 32 + h * 16 + it * 8 + (lane >> 3);
        gc = n0 + wcol + (lane & 7) * 8;
      };
      auto issue = [&](int n) {
        int lm, gc;
        pos(n, lm, gc);
        const bool ok = lm < m_valid && gc < p.N;
        // out-of-tile lanes read the tile's first valid element instead
        const int64_t o = static_cast<int64_t>(row0 + (ok ? lm : 0)) * p.ldh +
                          static_cast<int64_t>(ok ? gc : n0) * ES;
        q1[n].load(p.H1 + o);
        if constexpr (SW) q3[n].load(p.H3 + o);
      };
#pragma unroll
      for (int n = 0; n < kPf; ++n) issue(n);
#pragma unroll
      for (int n = 0; n < kIt; ++n) {
        if (n + kPf < kIt) issue(n + kPf);
        if ((n & 1) == 0) stage_strip(strip, acc, n >> 2, (n >> 1) & 1);
        int lm, gc;
        pos(n, lm, gc);
        if (lm < m_valid && gc < p.N) {
          const int r = (n & 1) * 8 + (lane >> 3), c8 = (lane & 7) * 8;
          const int64_t grow = row0 + lm;
          float h1[8], g1[8];
          q1[n].to_f(h1);
          if constexpr (SW) {
            float h3[8], g3[8];
            q3[n].to_f(h3);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              // d silu(h1) h3 / dh1 = h3 sg (1 + h1 (1 - sg)), d / dh3 = h1 sg
              const float da = strip[r * kStripPitch + c8 + e];
              const float sg = sigm(h1[e]);
              const float t = da * sg, u = t * h3[e];
              g1[e] = __builtin_fmaf(u, __builtin_fmaf(-h1[e], sg, h1[e]), u);
              g3[e] = t * h1[e];
            }
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(p.f + gc) * ES, g3);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              g1[e] = strip[r * kStripPitch + c8 + e] * act_grad_f(h1[e], p.act);
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
          }
        }
      }
    } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        stage_strip(strip, acc, i, h);
        const int srow0 = team * 128 + i * 32 + h * 16;  // strip's first row within the tile
        if constexpr (MODE == M_FWD1_SWIGLU) {
          // strip columns [0,32): H1, [32,64): H3 of hidden units n0 + 32wq + c
          const int r = lane >> 2, c8 = (lane & 3) * 8;
          const int lm = srow0 + r;
          const int gc = n0 + wq * 32 + c8;
          if (lm < m_valid && gc < p.N) {
            float h1[8], h3[8], a[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              h1[e] = Elem<T>::to_f(Elem<T>::from_f(strip[r * kStripPitch + c8 + e]));
              h3[e] = Elem<T>::to_f(Elem<T>::from_f(strip[r * kStripPitch + 32 + c8 + e]));
              a[e] = h1[e] * sigm(h1[e]) * h3[e];
            }
            const int64_t grow = row0 + lm;
            if (p.H1) {
              store_vec<T>(p.H1 + grow * p.ldh + static_cast<int64_t>(gc) * ES, h1);
              store_vec<T>(p.H3 + grow * p.ldh + static_cast<int64_t>(gc) * ES, h3);
            }
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, a);
          }
        } else if constexpr (MODE == M_FWD1 || MODE == M_STORE) {
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const int r = it * 8 + (lane >> 3), c8 = (lane & 7) * 8;
            const int lm = srow0 + r;
            const int gc = n0 + wcol + c8;
            if (lm < m_valid && gc < p.N) {
              float v[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) v[e] = strip[r * kStripPitch + c8 + e];
              const int64_t grow = row0 + lm;
              if constexpr (MODE == M_FWD1) {
                float hh[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  hh[e] = Elem<T>::to_f(Elem<T>::from_f(v[e]));
                  v[e] = act_f(hh[e], p.act);
                }
                if (p.H1) store_vec<T>(p.H1 + grow * p.ldh + static_cast<int64_t>(gc) * ES, hh);
              }
              store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, v);
            }
          }
        } else {  // M_DW: fp32 rows of dW (or of a partial-sum slot)
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const int r = it * 8 + (lane >> 3), c8 = (lane & 7) * 8;
            const int lm = srow0 + r;
            const int gc = n0 + wcol + c8;
            if (lm < m_valid && gc < p.N) {
              const int orow = row0 + lm;
              float* dst;
              if (slot >= 0) {
                dst = p.partial + static_cast<int64_t>(slot) * p.slot_elems +
                      static_cast<int64_t>(orow) * p.N + gc;
              } else if (orow < p.split_row) {
                dst = p.dwA + static_cast<int64_t>(g) * p.dw_gstride +
                      static_cast<int64_t>(orow) * p.N + gc;
              } else {
                dst = p.dwB + static_cast<int64_t>(g) * p.dw_gstride +
                      static_cast<int64_t>(orow - p.split_row) * p.N + gc;
              }
              const float* sp = strip + r * kStripPitch + c8;
              *reinterpret_cast<float4*>(dst) = make_float4(sp[0], sp[1], sp[2], sp[3]);
              *reinterpret_cast<float4*>(dst + 4) = make_float4(sp[4], sp[5], sp[6], sp[7]);
            }
          }
        }
      }
    }
    }
    __syncthreads();   // strips are free before the next tile's loads
  }
}

// ---------------------------------------------------------------------------
// fp32 forward products with few rows
// ---------------------------------------------------------------------------
// A 256x256 fp32 tile is one wavefront's 128x64 block on each of eight
// wavefronts, whatever the rows: with a few dozen rows per expert (fp32
// matrix cores run at a sixteenth of the bf16 rate) the handful of busy
// wavefronts sets the time.  Here one wavefront computes one 32x32 output
// block (gated: 32 hidden units of H1 and of H3) with v_mfma_f32_32x32x2f32,
// reading both K-contiguous operands straight from memory (64 k at a time,
// the next 64 in flight), so the work spreads over as many SIMDs as there
// are blocks.  Lane l supplies row (column) l % 32 and, for the four MFMAs
// of an 8-wide k step, k values k0 + 4 (l / 32) + j (j = 0..3): every k of
// the step enters exactly one MFMA, for the A and the B operand alike.  Item = (expert, 32-row block,
// 32-column block); blocks past the expert's rows or past N exit at once.
constexpr int kTinyB = 32;
constexpr int kTinyMaxItems = 4096;

template <int MODE>
__global__ __launch_bounds__(256) void ffn_gemm_f32_tiny_kernel(const GemmParams p, int E,
                                                                int mblocks, int nblocks) {
  constexpr bool GATED = MODE == M_FWD1_SWIGLU;
  const int lane = threadIdx.x & 63;
  const int item = static_cast<int>(blockIdx.x) * 4 + (static_cast<int>(threadIdx.x) >> 6);
  const int per_e = mblocks * nblocks;
  const int g = item / per_e;
  if (g >= E) return;
  const int rem = item - g * per_e;
  const int m0 = (rem / nblocks) * kTinyB, n0 = (rem % nblocks) * kTinyB;
  const int rows_g = p.sched->rows[g];
  if (m0 >= rows_g || n0 >= p.N) return;
  const int r = lane & 31, kh = 4 * (lane >> 5);
  const bool arow = m0 + r < rows_g, brow = n0 + r < p.N;
  const int64_t grow0 = static_cast<int64_t>(p.offsets[g]) + m0;
  const float* a = reinterpret_cast<const float*>(p.A + (grow0 + (arow ? r : 0)) * p.lda);
  const int64_t boff = static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0 + (brow ? r : 0)) * p.ldb;
  const float* b1 = reinterpret_cast<const float*>(p.B + boff);
  const float* b3 = GATED ? reinterpret_cast<const float*>(p.B2 + boff) : b1;
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  floatx16 c1, c3;
#pragma unroll
  for (int q = 0; q < 16; ++q) c1[q] = c3[q] = 0.f;
  // k in chunks of 64 (8 steps of 8): a chunk's operands are loaded
  // together, the next chunk's before the current chunk's MFMAs (K is a
  // multiple of 8; steps past K load zeros)
  constexpr int kSteps = 8;
  struct Chunk { float4 a[kSteps], b[kSteps], w[kSteps]; };
  auto load = [&](int k0, Chunk& c) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      const int kk = k0 + 8 * s + kh;
      const bool ok = kk < p.K;
      c.a[s] = arow && ok ? *reinterpret_cast<const float4*>(a + kk) : zero;
      c.b[s] = brow && ok ? *reinterpret_cast<const float4*>(b1 + kk) : zero;
      if constexpr (GATED) c.w[s] = brow && ok ? *reinterpret_cast<const float4*>(b3 + kk) : zero;
    }
  };
  auto mma = [&](const Chunk& c) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].x, c.b[s].x, c1, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].y, c.b[s].y, c1, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].z, c.b[s].z, c1, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].w, c.b[s].w, c1, 0, 0, 0);
      if constexpr (GATED) {
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].x, c.w[s].x, c3, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].y, c.w[s].y, c3, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].z, c.w[s].z, c3, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x2f32(c.a[s].w, c.w[s].w, c3, 0, 0, 0);
      }
    }
  };
  constexpr int KC = 8 * kSteps;
  Chunk c0, cn;
  load(0, c0);
  for (int k0 = 0; k0 < p.K; k0 += 2 * KC) {
    if (k0 + KC < p.K) load(k0 + KC, cn);
    mma(c0);
    if (k0 + KC >= p.K) break;
    if (k0 + 2 * KC < p.K) load(k0 + 2 * KC, c0);
    mma(cn);
  }
  // accumulator q of lane l: column l % 32, row 8 (q / 4) + 4 (l / 32) + q % 4
  const int col = n0 + r;
  if (col >= p.N) return;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int row = m0 + 8 * (q >> 2) + kh + (q & 3);
    if (row >= rows_g) continue;
    const int64_t grow = static_cast<int64_t>(p.offsets[g]) + row;
    float* cp = reinterpret_cast<float*>(p.C + grow * p.ldc) + col;
    if constexpr (MODE == M_FWD1_SWIGLU) {
      const float h1 = c1[q], h3 = c3[q];
      if (p.H1) {
        reinterpret_cast<float*>(p.H1 + grow * p.ldh)[col] = h1;
        reinterpret_cast<float*>(p.H3 + grow * p.ldh)[col] = h3;
      }
      *cp = h1 * sigm(h1) * h3;
    } else if constexpr (MODE == M_FWD1) {
      if (p.H1) reinterpret_cast<float*>(p.H1 + grow * p.ldh)[col] = c1[q];
      *cp = act_f(c1[q], p.act);
    } else {
      *cp = c1[q];
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 products: four wavefronts of 128x128
// ---------------------------------------------------------------------------
// bf16 layers run every product on 4 wavefronts, one per SIMD, each holding a
// 128x128 block of the 256x256 tile as 64 blocks of 16x16 fp32 accumulators
// (v_mfma_f32_16x16x32_bf16, 256 accumulation registers).  Per K step of 64
// there are two barriers, one after the A and one after the B fragment reads
// of the step's stage.  Between the MFMAs each wave issues, one at a time,
// the fragment reads of the next half step and, once a barrier has freed its
// part of the stage, its share of the direct-to-LDS loads of the step after
// next, so the memory pipeline sees a steady stream of requests while the
// matrix core stays busy.  A 128x128 block reads a third less LDS per MFMA
// than a 128x64 one.
constexpr int kThreads16 = 256;

typedef int intx4 __attribute__((ext_vector_type(4)));

// c += a * b for one 16x16 block.  Lane l = 16 G + c16 supplies row c16 of
// the A and B sub-blocks at k = 8 G .. 8 G + 7 and holds rows 4 G .. 4 G + 3,
// column c16 of the result.  Inline assembly keeps each accumulator in place
// in its accumulation registers through the K loop (compiled MFMAs get their
// accumulators shuffled between loop iterations).  Consecutive updates of one
// accumulator are at least 63 MFMAs apart, and the fragments an MFMA reads
// are not rewritten for at least 28 MFMAs, so no wait states are needed
// inside the loop; the epilogue waits before it reads the accumulators.
__device__ __forceinline__ void mfma16(floatx4& c, const uint4& a, const uint4& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
               : "+a"(c)
               : "v"(__builtin_bit_cast(intx4, a)), "v"(__builtin_bit_cast(intx4, b)));
}

// acc += A_tile * B_tile^T over the whole K extent (see above).  Wave w owns
// tile rows 128 (w >> 1) .. +127 and columns 128 (w & 1) .. +127 (gated
// forward: hidden units 64 (w & 1) .. +63 of W1, then the same units of W3).
// The four stage objects are distinct, and the loop is unrolled by two so
// every LDS access names its object statically: the compiler can then tell
// the loads into one stage from the reads of the other.
template <int ALAY, int BLAY, bool GATED, bool FULL>
__device__ __forceinline__ void mainloop16(const TileOps& op, char* la0, char* lb0, char* la1,
                                           char* lb1, floatx4 (&acc)[8][8], int zt) {
  constexpr int KSTEP = 64;
  const int lane = (static_cast<int>(threadIdx.x) & 63) + zt;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int K = op.K;
  const int nk = (K + KSTEP - 1) / KSTEP;
  if (nk <= 0) return;
  const int nk2 = (nk + 1) & ~1;   // odd counts load one all-zero step

  // ---- loads: 1 KB blocks (8 rows of a KC tile: lane l -> row l >> 3,
  // physical chunk l & 7; or 2 k-rows of a KM tile: lane l -> k-row l >> 5,
  // physical elements 8 (l & 31) .. +7); wave w loads blocks 8w .. 8w+7 of
  // A (g = 0..7) and of B (g = 8..15) of every stage.
  const int l3 = lane >> 3;
  const int co0 = ((lane & 7) ^ swz(l3)) * 16, co1 = ((lane & 7) ^ swz(l3 + 8)) * 16;
  const int kr = lane >> 5;            // KM: k-row within the block
  const int pe = (lane & 31) * 8;      // KM: physical element within the k-row
  auto km_col = [&](int q) { return (((pe >> 5) ^ q) << 5) + (pe & 31); };
  const __amdgpu_buffer_rsrc_t ra_t = tile_rsrc(op.a.base);
  const __amdgpu_buffer_rsrc_t rb_t = tile_rsrc(op.b.base);
  const __amdgpu_buffer_rsrc_t rb3_t = tile_rsrc(GATED ? op.b.base2 : op.b.base);
  auto km_rsrc = [&](const Operand& o, int kt, bool second) {
    const int64_t k = static_cast<int64_t>(kt) * KSTEP - (second ? o.split : 0);
    return tile_rsrc((second ? o.base2 : o.base) + k * o.ld);
  };
  // the resources and flags of one K step, set once per step
  struct StepLd {
    __amdgpu_buffer_rsrc_t ra, ra2, rb, rb2;
    int kt;
    bool kfull, kany;
  };
  auto step_ld = [&](int kt) {
    StepLd s;
    s.kt = kt;
    s.kfull = (kt + 1) * KSTEP <= K;
    s.kany = kt * KSTEP < K;
    s.ra = ra_t; s.ra2 = ra_t; s.rb = rb_t; s.rb2 = rb3_t;
    if constexpr (ALAY == L_KM) {
      s.ra = km_rsrc(op.a, kt, false);
      s.ra2 = op.a.base2 ? km_rsrc(op.a, kt, true) : s.ra;
    }
    if constexpr (BLAY == L_KM) {
      s.rb = km_rsrc(op.b, kt, false);
      s.rb2 = op.b.base2 ? km_rsrc(op.b, kt, true) : s.rb;
    }
    return s;
  };
  // block blk of operand o (layout LAY) of step s.kt into dst
  auto load_blk = [&](auto lay, const Operand& o, const __amdgpu_buffer_rsrc_t& rs,
                      const __amdgpu_buffer_rsrc_t& rs2, char* dst, int blk, const StepLd& s,
                      bool gated) {
    constexpr int LAY = decltype(lay)::value;
    const int ld = static_cast<int>(o.ld);
    uint32_t off;
    int soff;
    bool second = false;
    if constexpr (LAY == L_KC) {
      const int co = (blk & 1) ? co1 : co0;
      // gated forward: 64-row groups alternate W1 / W3 rows of 64 hidden units
      const int row0 = gated ? (blk >> 4) * 64 + (blk & 7) * 8 : blk * 8;
      second = gated && ((blk >> 3) & 1);
      off = static_cast<uint32_t>(l3 * ld) + co;
      soff = row0 * ld + s.kt * kRowBytes;
      if (!FULL || !s.kfull) {
        const bool ok = (FULL || row0 + l3 < o.rows) && (s.kfull || s.kt * kRowBytes + co < K * 2);
        if (!ok) off = kOob;
      }
    } else {
      const int krel = 2 * blk;                  // first k-row of the block in the step
      const int kabs = s.kt * KSTEP + krel;
      const int q = (krel + kr) & 3;
      const int col = km_col(q);
      second = kabs >= o.split;
      off = static_cast<uint32_t>(kr * ld + col * 2);
      soff = krel * ld;
      if (!FULL || !s.kfull) {
        const bool ok = (FULL || col < o.rows) && (s.kfull || kabs + kr < K);
        if (!ok) off = kOob;
      }
    }
    if (!s.kany) off = kOob;
    if (second)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
  };
  using KC_ = std::integral_constant<int, L_KC>;
  using KM_ = std::integral_constant<int, L_KM>;
  // one of the wave's 16 loads of a stage
  auto load1 = [&](const StepLd& s, char* sa, char* sb, int g) {
    const int blk = wave * 8 + (g & 7);
    if (g < 8) {
      if constexpr (ALAY == L_KC) load_blk(KC_{}, op.a, s.ra, s.ra2, sa, blk, s, false);
      else load_blk(KM_{}, op.a, s.ra, s.ra2, sa, blk, s, false);
    } else {
      if constexpr (BLAY == L_KC) load_blk(KC_{}, op.b, s.rb, s.rb2, sb, blk, s, GATED);
      else load_blk(KM_{}, op.b, s.rb, s.rb2, sb, blk, s, false);
    }
  };

  // ---- fragments.  KC: lane l = 16 G + c16 reads row c16 of a 16-row block,
  // logical chunk 4h + G (k = 32h + 8G .. +7) of the 128-byte row; the row's
  // swizzle is (c16 >> 1) since blocks start at multiples of 16.
  const int c16 = lane & 15, G = lane >> 4;
  const int fa_kc = (wm * 128 + c16) * kRowBytes, fb_kc = (wn * 128 + c16) * kRowBytes;
  // KM: two transpose reads, k-rows 32h + 8G + (c16 >> 2) and 4 below, columns
  // cb + 4 (c16 & 3) .. +3 (lane 4a + b of a 16-lane group then holds column
  // cb + 4a + b at 4 consecutive k); segment swizzle by k & 3 = c16 >> 2
  auto km_frag = [&](const char* st, int cb, int h) -> uint4 {
    const int phys = (((cb >> 5) ^ (c16 >> 2)) << 5) + (cb & 31) + 4 * (c16 & 3);
    const char* p0 = st + (32 * h + 8 * G + (c16 >> 2)) * 512 + phys * 2;
    const uint2 lo = read_tr(p0);
    const uint2 hi = read_tr(p0 + 4 * 512);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  };
  // fragment g of half h: A sub-block g (g < 8) or B sub-block g - 8
  auto read1 = [&](const char* sa, const char* sb, int h, uint4 (&fa)[8], uint4 (&fb)[8], int g) {
    const int sw = ((4 * h + G) ^ (c16 >> 1)) << 4;
    if (g < 8) {
      if constexpr (ALAY == L_KC)
        fa[g] = *reinterpret_cast<const uint4*>(sa + fa_kc + g * 16 * kRowBytes + sw);
      else
        fa[g] = km_frag(sa, wm * 128 + g * 16, h);
    } else {
      if constexpr (BLAY == L_KC)
        fb[g - 8] = *reinterpret_cast<const uint4*>(sb + fb_kc + (g - 8) * 16 * kRowBytes + sw);
      else
        fb[g - 8] = km_frag(sb, wn * 128 + (g - 8) * 16, h);
    }
  };
  uint4 f0a[8], f0b[8], f1a[8], f1b[8];   // fragments of k-half 0 / 1 of a stage

  // Every wave runs the same instruction stream on every tile: rows, columns
  // and K past the valid ones were loaded as zeros, so a wave with no valid
  // rows or columns multiplies zeros, and the epilogue stores none of them.
  // (Skipping such a wave's reads and MFMAs with a branch per group broke
  // the interleaving for the whole tile: a partial tile then took several
  // times as long as a full one.)

  // One K step from stage (ca, cb), the next stage in (na, nb); the loads of
  // step kt + 2 go into (ca, cb): its A part once every wave has read the A
  // fragments of k-half 1, its B part once every wave has read the B ones.
  // Two barriers per step let the 16 loads spread over the last three
  // quarters of the step (one per 6 MFMAs) instead of crowding into the
  // second half.
  auto step = [&](int kt, char* ca, char* cb, const char* na, const char* nb) {
    const StepLd s = step_ld(kt + 2);
    // first quarter: MFMAs 0..31 of k-half 0, reads of the A fragments of k-half 1
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      read1(ca, cb, 1, f1a, f1b, g);
#pragma unroll
      for (int m = 4 * g; m < 4 * g + 4; ++m) mfma16(acc[m >> 3][m & 7], f0a[m >> 3], f0b[m & 7]);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // second quarter: MFMAs 32..63 of k-half 0, reads of the B fragments of
    // k-half 1, the A loads of step kt + 2
#pragma unroll
    for (int g = 8; g < 16; ++g) {
      // A loads 0..5 at groups 8, 9, 11, 12, 14, 15
      if (g % 3 != 1) load1(s, ca, cb, g - 8 - (g - 8) / 3);
      read1(ca, cb, 1, f1a, f1b, g);
#pragma unroll
      for (int m = 4 * g; m < 4 * g + 4; ++m) mfma16(acc[m >> 3][m & 7], f0a[m >> 3], f0b[m & 7]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // stage kt + 1 has landed (only the 6 A loads just issued may be pending)
    __builtin_amdgcn_s_waitcnt(0x0076);   // vmcnt(6) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // second half: MFMAs of k-half 1, reads of the next stage's k-half 0, the
    // B loads of step kt + 2
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      // A loads 6, 7 and the B loads at groups 0, 2, 3, 5, 6, 8, 9, 11, 12, 14
      if (g % 3 != 1 && g < 15) load1(s, ca, cb, 6 + g - (g + 1) / 3);
      read1(na, nb, 0, f0a, f0b, g);
#pragma unroll
      for (int m = 4 * g; m < 4 * g + 4; ++m) mfma16(acc[m >> 3][m & 7], f1a[m >> 3], f1b[m & 7]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  {
    const StepLd s0 = step_ld(0), s1 = step_ld(1);
#pragma unroll
    for (int g = 0; g < 16; ++g) load1(s0, la0, lb0, g);
#pragma unroll
    for (int g = 0; g < 16; ++g) load1(s1, la1, lb1, g);
  }
  __builtin_amdgcn_s_waitcnt(0x4F70);   // vmcnt(16): this wave's stage-0 loads landed
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int g = 0; g < 16; ++g) read1(la0, lb0, 0, f0a, f0b, g);
  for (int kt = 0; kt < nk2; kt += 2) {
    step(kt, la0, lb0, la1, lb1);
    step(kt + 1, la1, lb1, la0, lb0);
  }
  __builtin_amdgcn_s_waitcnt(0x0070);
  __builtin_amdgcn_s_barrier();   // every load landed, every read done: stages are free
  // the epilogue reads the accumulators with ordinary instructions
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// ---------------------------------------------------------------------------
// bf16 products on 128x128 tiles, two workgroups per CU
// ---------------------------------------------------------------------------
// The 256x256 kernel holds one wavefront per SIMD (256 accumulation
// registers), so a tile's prologue and epilogue leave the matrix cores idle:
// on short K (a few K steps per tile), few tiles per CU, or an epilogue heavy
// in VALU work, that idle time is a large share.  This variant computes
// 128x128 tiles with 4 wavefronts of 64x64 (64 accumulation registers,
// under 256 registers in all) and 64 KB of LDS, so two workgroups share each
// CU and one's epilogue overlaps the other's MFMAs.  It reads twice the
// operand bytes per flop of the 256x256 tile, which is why large products
// keep the big tile.  The K loop has the same structure: two stages of K 64,
// two barriers per step, and loads and fragment reads issued one at a time
// between the MFMAs.
//
// Wave w owns tile rows 64 (w >> 1) .. +63 and columns 64 (w & 1) .. +63
// (gated forward: hidden units 32 (w & 1) .. +31 of W1, then the same units
// of W3).  KC LDS tiles are 128 rows of 128 bytes with the swizzle of the
// big tile; KM tiles are 64 k-rows of 128 elements (256 bytes) with the
// same XOR of 32-element segments by k mod 4.
template <int ALAY, int BLAY, bool GATED, bool FULL>
__device__ __forceinline__ void mainloop16s(const TileOps& op, char* la0, char* lb0, char* la1,
                                            char* lb1, floatx4 (&acc)[4][4], int zt) {
  constexpr int KSTEP = 64;
  constexpr int KMROW = 256;           // bytes per k-row of a KM tile
  const int lane = (static_cast<int>(threadIdx.x) & 63) + zt;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int K = op.K;
  const int nk = (K + KSTEP - 1) / KSTEP;
  if (nk <= 0) return;
  const int nk2 = (nk + 1) & ~1;   // odd counts load one all-zero step

  // ---- loads: 1 KB blocks (8 rows of a KC tile: lane l -> row l >> 3,
  // physical chunk l & 7; or 4 k-rows of a KM tile: lane l -> k-row l >> 4,
  // physical elements 8 (l & 15) .. +7); wave w loads blocks 4w .. 4w+3 of
  // A (g = 0..3) and of B (g = 4..7) of every stage.
  const int l3 = lane >> 3;
  const int co0 = ((lane & 7) ^ swz(l3)) * 16, co1 = ((lane & 7) ^ swz(l3 + 8)) * 16;
  const int kr = lane >> 4;            // KM: k-row within the block (= k mod 4)
  const int pe = (lane & 15) * 8;      // KM: physical element within the k-row
  const int km_col = (((pe >> 5) ^ kr) << 5) + (pe & 31);
  const __amdgpu_buffer_rsrc_t ra_t = tile_rsrc(op.a.base);
  const __amdgpu_buffer_rsrc_t rb_t = tile_rsrc(op.b.base);
  const __amdgpu_buffer_rsrc_t rb3_t = tile_rsrc(GATED ? op.b.base2 : op.b.base);
  auto km_rsrc = [&](const Operand& o, int kt, bool second) {
    const int64_t k = static_cast<int64_t>(kt) * KSTEP - (second ? o.split : 0);
    return tile_rsrc((second ? o.base2 : o.base) + k * o.ld);
  };
  struct StepLd {
    __amdgpu_buffer_rsrc_t ra, ra2, rb, rb2;
    int kt;
    bool kfull, kany;
  };
  auto step_ld = [&](int kt) {
    StepLd s;
    s.kt = kt;
    s.kfull = (kt + 1) * KSTEP <= K;
    s.kany = kt * KSTEP < K;
    s.ra = ra_t; s.ra2 = ra_t; s.rb = rb_t; s.rb2 = rb3_t;
    if constexpr (ALAY == L_KM) {
      s.ra = km_rsrc(op.a, kt, false);
      s.ra2 = op.a.base2 ? km_rsrc(op.a, kt, true) : s.ra;
    }
    if constexpr (BLAY == L_KM) {
      s.rb = km_rsrc(op.b, kt, false);
      s.rb2 = op.b.base2 ? km_rsrc(op.b, kt, true) : s.rb;
    }
    return s;
  };
  auto load_blk = [&](auto lay, const Operand& o, const __amdgpu_buffer_rsrc_t& rs,
                      const __amdgpu_buffer_rsrc_t& rs2, char* dst, int blk, const StepLd& s,
                      bool gated) {
    constexpr int LAY = decltype(lay)::value;
    const int ld = static_cast<int>(o.ld);
    uint32_t off;
    int soff;
    bool second = false;
    if constexpr (LAY == L_KC) {
      const int co = (blk & 1) ? co1 : co0;
      // gated forward: 32-row groups alternate W1 / W3 rows of 32 hidden units
      const int row0 = gated ? (blk >> 3) * 32 + (blk & 3) * 8 : blk * 8;
      second = gated && ((blk >> 2) & 1);
      off = static_cast<uint32_t>(l3 * ld) + co;
      soff = row0 * ld + s.kt * kRowBytes;
      if (!FULL || !s.kfull) {
        const bool ok = (FULL || row0 + l3 < o.rows) && (s.kfull || s.kt * kRowBytes + co < K * 2);
        if (!ok) off = kOob;
      }
    } else {
      const int krel = 4 * blk;                  // first k-row of the block in the step
      const int kabs = s.kt * KSTEP + krel;
      second = kabs >= o.split;                  // split is a multiple of 8: no block straddles it
      off = static_cast<uint32_t>(kr * ld + km_col * 2);
      soff = krel * ld;
      if (!FULL || !s.kfull) {
        const bool ok = (FULL || km_col < o.rows) && (s.kfull || kabs + kr < K);
        if (!ok) off = kOob;
      }
    }
    if (!s.kany) off = kOob;
    if (second)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, MOE_LDS(dst + blk * 1024), 16, off, soff, 0, 0);
  };
  using KC_ = std::integral_constant<int, L_KC>;
  using KM_ = std::integral_constant<int, L_KM>;
  auto load1 = [&](const StepLd& s, char* sa, char* sb, int g) {
    const int blk = wave * 4 + (g & 3);
    if (g < 4) {
      if constexpr (ALAY == L_KC) load_blk(KC_{}, op.a, s.ra, s.ra2, sa, blk, s, false);
      else load_blk(KM_{}, op.a, s.ra, s.ra2, sa, blk, s, false);
    } else {
      if constexpr (BLAY == L_KC) load_blk(KC_{}, op.b, s.rb, s.rb2, sb, blk, s, GATED);
      else load_blk(KM_{}, op.b, s.rb, s.rb2, sb, blk, s, false);
    }
  };

  // ---- fragments (as in the 256x256 kernel; KM k-rows are 256 bytes)
  const int c16 = lane & 15, G = lane >> 4;
  const int fa_kc = (wm * 64 + c16) * kRowBytes, fb_kc = (wn * 64 + c16) * kRowBytes;
  auto km_frag = [&](const char* st, int cb, int h) -> uint4 {
    const int phys = (((cb >> 5) ^ (c16 >> 2)) << 5) + (cb & 31) + 4 * (c16 & 3);
    const char* p0 = st + (32 * h + 8 * G + (c16 >> 2)) * KMROW + phys * 2;
    const uint2 lo = read_tr(p0);
    const uint2 hi = read_tr(p0 + 4 * KMROW);
    return make_uint4(lo.x, lo.y, hi.x, hi.y);
  };
  // fragment g of half h: A sub-block g (g < 4) or B sub-block g - 4
  auto read1 = [&](const char* sa, const char* sb, int h, uint4 (&fa)[4], uint4 (&fb)[4], int g) {
    const int sw = ((4 * h + G) ^ (c16 >> 1)) << 4;
    if (g < 4) {
      if constexpr (ALAY == L_KC)
        fa[g] = *reinterpret_cast<const uint4*>(sa + fa_kc + g * 16 * kRowBytes + sw);
      else
        fa[g] = km_frag(sa, wm * 64 + g * 16, h);
    } else {
      if constexpr (BLAY == L_KC)
        fb[g - 4] = *reinterpret_cast<const uint4*>(sb + fb_kc + (g - 4) * 16 * kRowBytes + sw);
      else
        fb[g - 4] = km_frag(sb, wn * 64 + (g - 4) * 16, h);
    }
  };
  uint4 f0a[4], f0b[4], f1a[4], f1b[4];

  // One K step from stage (ca, cb), the next stage in (na, nb); the loads of
  // step kt + 2 go into (ca, cb).  MFMAs in groups of two (m -> block
  // m >> 2, m & 3); the first quarter reads the A fragments of k-half 1, the
  // second the B fragments and issues the A loads, the second half reads the
  // next stage's k-half 0 and issues the B loads.
  auto step = [&](int kt, char* ca, char* cb, const char* na, const char* nb) {
    const StepLd s = step_ld(kt + 2);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      read1(ca, cb, 1, f1a, f1b, g);
#pragma unroll
      for (int m = 2 * g; m < 2 * g + 2; ++m) mfma16(acc[m >> 2][m & 3], f0a[m >> 2], f0b[m & 3]);
      __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int g = 4; g < 8; ++g) {
      load1(s, ca, cb, g - 4);
      read1(ca, cb, 1, f1a, f1b, g);
#pragma unroll
      for (int m = 2 * g; m < 2 * g + 2; ++m) mfma16(acc[m >> 2][m & 3], f0a[m >> 2], f0b[m & 3]);
      __builtin_amdgcn_sched_barrier(0);
    }
    // stage kt + 1 has landed (only the 4 A loads just issued may be pending)
    __builtin_amdgcn_s_waitcnt(0x0074);   // vmcnt(4) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      if ((g & 1) == 0) load1(s, ca, cb, 4 + (g >> 1));
      read1(na, nb, 0, f0a, f0b, g);
#pragma unroll
      for (int m = 2 * g; m < 2 * g + 2; ++m) mfma16(acc[m >> 2][m & 3], f1a[m >> 2], f1b[m & 3]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  {
    const StepLd s0 = step_ld(0), s1 = step_ld(1);
#pragma unroll
    for (int g = 0; g < 8; ++g) load1(s0, la0, lb0, g);
#pragma unroll
    for (int g = 0; g < 8; ++g) load1(s1, la1, lb1, g);
  }
  __builtin_amdgcn_s_waitcnt(0x0F78);   // vmcnt(8): this wave's stage-0 loads landed
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int g = 0; g < 8; ++g) read1(la0, lb0, 0, f0a, f0b, g);
  for (int kt = 0; kt < nk2; kt += 2) {
    step(kt, la0, lb0, la1, lb1);
    step(kt + 1, la1, lb1, la0, lb0);
  }
  __builtin_amdgcn_s_waitcnt(0x0070);
  __builtin_amdgcn_s_barrier();   // every load landed, every read done: stages are free
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// Wave-block shapes of the two bf16 kernels: RB x CB blocks of 16x16 per
// wave, 2 x 2 waves per workgroup.
template <int RB_, int CB_, int MINB_> struct Tile16 {
  static constexpr int RB = RB_, CB = CB_;
  static constexpr int WR = 16 * RB, WC = 16 * CB;      // wave block
  static constexpr int TM = 2 * WR, TN = 2 * WC;        // workgroup tile
  static constexpr int kP = WC + 4;                     // strip pitch (floats): rows 4 apart
                                                        // fall 16 banks apart
  static constexpr int kStripBytes = 16 * kP * 4;
  static constexpr int kStageBytes = TM * kRowBytes;    // one operand of one stage
  static constexpr int kMinBlocks = MINB_;              // workgroups per CU
  static_assert(2 * kStripBytes <= kStageBytes, "two staging strips per operand buffer");
};
using TileBig = Tile16<8, 8, 1>;
using TileSmall = Tile16<4, 4, 2>;
static_assert(TileBig::TM == BM && TileBig::TN == BN && TileSmall::TM == BM_S, "tile sizes");

// Stage rows 16i .. 16i+15 of the wave's accumulators as fp32, row pitch C::kP.
template <typename C>
__device__ __forceinline__ void stage16(float* strip, const floatx4 (&acc)[C::RB][C::CB], int i,
                                        int lane) {
  const int c16 = lane & 15, G = lane >> 4;
#pragma unroll
  for (int j = 0; j < C::CB; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) strip[(4 * G + q) * C::kP + 16 * j + c16] = acc[i][j][q];
}

template <int MODE, int PASS, typename C>
__global__ __launch_bounds__(kThreads16, C::kMinBlocks) void ffn_gemm16_kernel(const GemmParams p) {
  __shared__ __attribute__((aligned(16))) char la0[C::kStageBytes];
  __shared__ __attribute__((aligned(16))) char lb0[C::kStageBytes];
  __shared__ __attribute__((aligned(16))) char la1[C::kStageBytes];
  __shared__ __attribute__((aligned(16))) char lb1[C::kStageBytes];
  constexpr bool SMALL = C::RB == 4;
  constexpr int TM = C::TM, TN = C::TN, WR = C::WR, WC = C::WC, kP = C::kP;
  using T = uint16_t;
  constexpr int ES = 2;
  constexpr bool VARK = MODE == M_DW;
  constexpr bool GATED = MODE == M_FWD1_SWIGLU;
  constexpr int ALAY = a_layout(PASS), BLAY = b_layout(PASS);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const Sched& sc = *p.sched;
  const int n_mt = SMALL ? sc.n_mtiles_s : sc.n_mtiles;
  const int n_items = VARK ? sc.n_segs * p.mtiles_out * p.ntiles : n_mt * p.ntiles;
  const int G = gridDim.x;
  const int lbase = (blockIdx.x % kXcds) * (G / kXcds) + blockIdx.x / kXcds;

  for (int round = 0;; ++round) {
    const int L = round * G + lbase;
    if (L >= n_items) break;
    TileOps op;
    int g, row0, m_valid, n0;
    int slot = -1, mt, nt;
    if constexpr (!VARK) {
      int mti;
      decode_banded(L, n_mt, p.ntiles, mti, nt);
      const int2 tm = p.mtile[mti];
      g = tm.x;
      row0 = p.offsets[g] + tm.y;
      m_valid = min(TM, sc.rows[g] - tm.y);
      op.a = {p.A + static_cast<int64_t>(row0) * p.lda, nullptr, p.lda, m_valid, 0};
      op.K = p.K;
      const char* bg = p.B + static_cast<int64_t>(g) * p.b_gstride;
      if constexpr (GATED) {
        n0 = nt * (TN / 2);
        op.b = {bg + static_cast<int64_t>(n0) * p.ldb,
                p.B2 + static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0) * p.ldb,
                p.ldb, min(TN / 2, p.N - n0), 0};
      } else if constexpr (BLAY == L_KC) {
        n0 = nt * TN;
        op.b = {bg + static_cast<int64_t>(n0) * p.ldb, nullptr, p.ldb, min(TN, p.N - n0), 0};
      } else {
        n0 = nt * TN;
        op.b = {bg + static_cast<int64_t>(n0) * ES,
                p.B2 ? p.B2 + static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0) * ES
                     : nullptr,
                p.ldb, min(TN, p.N - n0), p.B2 ? p.kmsplit : 0x7FFFFFFF};
      }
    } else {
      const int tmn = p.mtiles_out * p.ntiles;
      const int si = L / tmn;
      decode_banded(L - si * tmn, p.mtiles_out, p.ntiles, mt, nt);
      const int4 sg = p.seg[si];
      g = sg.x;
      slot = sg.w;
      const int k1 = min(sg.z, sc.rows[g]);
      const int64_t krow = static_cast<int64_t>(p.offsets[g]) + sg.y;
      row0 = mt * TM;
      n0 = nt * TN;
      m_valid = min(TM, p.M_out - row0);
      op.a = {p.A + krow * p.lda + static_cast<int64_t>(row0) * ES, nullptr, p.lda, m_valid,
              0x7FFFFFFF};
      op.b = {p.B + krow * p.ldb + static_cast<int64_t>(n0) * ES, nullptr, p.ldb,
              min(TN, p.N - n0), 0x7FFFFFFF};
      op.K = max(0, k1 - sg.y);
    }

    // the main loop derives its per-lane constants from an opaque zero made
    // per tile, so they are recomputed per tile instead of being hoisted out
    // of the tile loop and spilled (their reloads would wait on the loads)
    int zt;
    asm volatile("s_mov_b32 %0, 0" : "=s"(zt));
    floatx4 acc[C::RB][C::CB];
    const bool full = op.a.rows >= TM && op.b.rows >= (GATED ? TN / 2 : TN);
    if constexpr (SMALL) {
      if (full) mainloop16s<ALAY, BLAY, GATED, true>(op, la0, lb0, la1, lb1, acc, zt);
      else mainloop16s<ALAY, BLAY, GATED, false>(op, la0, lb0, la1, lb1, acc, zt);
    } else {
      if (full) mainloop16<ALAY, BLAY, GATED, true>(op, la0, lb0, la1, lb1, acc, zt);
      else mainloop16<ALAY, BLAY, GATED, false>(op, la0, lb0, la1, lb1, acc, zt);
    }

    // Epilogue, wave by wave: 16 accumulator rows at a time go through the
    // wave's LDS strip; a lane then finishes 8 consecutive columns of a row
    // and writes them as one vector (bf16) or two (fp32 weight gradients).
    // The lane index and the strip address are derived from an opaque zero
    // produced here, so nothing the epilogue computes per lane is hoisted
    // and held in registers across the K loop.
    int z;
    asm volatile("s_mov_b32 %0, 0" : "=s"(z));
    const int el = lane + z;
    float* strip = reinterpret_cast<float*>((wave < 2 ? la0 : lb0) + (wave & 1) * C::kStripBytes + z);
    const int wr0 = wm * WR;                      // the wave's first tile row
    // weight gradients: where the fp32 result of tile row orow, column gc goes
    // (a split partial-sum slot, or the first or second gradient array)
    auto dw_dst = [&](int orow, int gc) -> float* {
      if (slot >= 0)
        return p.partial + static_cast<int64_t>(slot) * p.slot_elems +
               static_cast<int64_t>(orow) * p.N + gc;
      if (orow < p.split_row)
        return p.dwA + static_cast<int64_t>(g) * p.dw_gstride + static_cast<int64_t>(orow) * p.N + gc;
      return p.dwB + static_cast<int64_t>(g) * p.dw_gstride +
             static_cast<int64_t>(orow - p.split_row) * p.N + gc;
    };
    if constexpr (VARK) {
      if (op.K == 0) {
        // no rows to contract over (an expert without rows): the tile is
        // zero; each lane stores 8 zeros per row pass straight to memory,
        // with no staging, so the tile costs only its stores.  Every wave
        // of the workgroup takes this path, and none touched the LDS.
        constexpr int LR = WC / 8, RG = 64 / LR;
        const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
        for (int r = 0; r < WR; r += RG) {
          const int lm = wr0 + r + el / LR, gc = n0 + wn * WC + (el % LR) * 8;
          if (lm < m_valid && gc < p.N) {
            float* dst = dw_dst(row0 + lm, gc);
            *reinterpret_cast<float4*>(dst) = zero;
            *reinterpret_cast<float4*>(dst + 4) = zero;
          }
        }
        continue;
      }
    }
    // ReLU / GELU layers: the epilogue is specialised on the activation, one
    // uniform branch per tile instead of one per element
    auto epilogue = [&](auto act_c) {
    constexpr int ACT = decltype(act_c)::value;
    if constexpr (MODE == M_FWD1_SWIGLU) {
      // strip columns [0,U): H1, [U,2U): H3 of hidden units n0 + U wn + u, U =
      // WC / 2; LU lanes cover a row's U units, 8 each
      constexpr int U = WC / 2, LU = U / 8, RU = 64 / LU;
#pragma unroll
      for (int i = 0; i < C::RB; ++i) {
        stage16<C>(strip, acc, i, el);
#pragma unroll
        for (int it = 0; it < 16 / RU; ++it) {
          const int r = it * RU + el / LU, u8 = (el % LU) * 8;
          const int lm = wr0 + 16 * i + r;
          const int gc = n0 + wn * U + u8;
          if (lm < m_valid && gc < p.N) {
            // H1 and H3 rounded to bf16 once: the packed bits are stored and
            // their values feed the activation
            float h1[8], h3[8], a[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              h1[e] = strip[r * kP + u8 + e];
              h3[e] = strip[r * kP + U + u8 + e];
            }
            const uint4 b1 = pack8(h1), b3 = pack8(h3);
            unpack8(b1, h1);
            unpack8(b3, h3);
#pragma unroll
            for (int e = 0; e < 8; ++e) a[e] = h1[e] * sigm(h1[e]) * h3[e];
            const int64_t grow = row0 + lm;
            if (p.H1) {
              *reinterpret_cast<uint4*>(p.H1 + grow * p.ldh + static_cast<int64_t>(gc) * ES) = b1;
              *reinterpret_cast<uint4*>(p.H3 + grow * p.ldh + static_cast<int64_t>(gc) * ES) = b3;
            }
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, a);
          }
        }
      }
    } else if constexpr (MODE == M_BWD_DA || MODE == M_BWD_DA_SWIGLU) {
      // dH = dA act'(H): (row block, row group) iterations, each reading 8
      // saved pre-activations (two planes for SwiGLU) per lane, issued kPf
      // iterations ahead of their use into a ring of kPf + 1 registers.  LR
      // lanes cover a row of the wave block, RG rows form a group, GB groups
      // a 16-row block.
      constexpr bool SW = MODE == M_BWD_DA_SWIGLU;
      constexpr int LR = WC / 8, RG = 64 / LR, GB = 16 / RG;
      constexpr int kIt = C::RB * GB, kPf = 4, kRing = kPf + 1;
      Raw8<T> q1[kRing], q3[kRing];
      auto pos = [&](int n, int& lm, int& gc) {
        lm = wr0 + 16 * (n / GB) + RG * (n % GB) + el / LR;
        gc = n0 + wn * WC + (el % LR) * 8;
      };
      auto issue = [&](int n) {
        int lm, gc;
        pos(n, lm, gc);
        const bool ok = lm < m_valid && gc < p.N;
        // out-of-tile lanes read the tile's first valid element instead
        const int64_t o = static_cast<int64_t>(row0 + (ok ? lm : 0)) * p.ldh +
                          static_cast<int64_t>(ok ? gc : n0) * ES;
        q1[n % kRing].load(p.H1 + o);
        if constexpr (SW) q3[n % kRing].load(p.H3 + o);
      };
#pragma unroll
      for (int n = 0; n < kPf; ++n) issue(n);
#pragma unroll
      for (int n = 0; n < kIt; ++n) {
        if (n + kPf < kIt) issue(n + kPf);
        if (n % GB == 0) stage16<C>(strip, acc, n / GB, el);
        int lm, gc;
        pos(n, lm, gc);
        if (lm < m_valid && gc < p.N) {
          const int r = RG * (n % GB) + el / LR, c8 = (el % LR) * 8;
          const int64_t grow = row0 + lm;
          float h1[8], g1[8];
          q1[n % kRing].to_f(h1);
          if constexpr (SW) {
            float h3[8], g3[8];
            q3[n % kRing].to_f(h3);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              // d silu(h1) h3 / dh1 = h3 sg (1 + h1 (1 - sg)), d / dh3 = h1 sg
              const float da = strip[r * kP + c8 + e];
              const float sg = sigm(h1[e]);
              const float t = da * sg, u = t * h3[e];
              g1[e] = __builtin_fmaf(u, __builtin_fmaf(-h1[e], sg, h1[e]), u);
              g3[e] = t * h1[e];
            }
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(p.f + gc) * ES, g3);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              g1[e] = strip[r * kP + c8 + e] * act_grad_f(h1[e], ACT);
            store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
          }
        }
      }
    } else {
      constexpr int LR = WC / 8, RG = 64 / LR;   // lanes per row, rows per pass
#pragma unroll
      for (int i = 0; i < C::RB; ++i) {
        stage16<C>(strip, acc, i, el);
#pragma unroll
        for (int it = 0; it < 16 / RG; ++it) {
          const int r = RG * it + el / LR, c8 = (el % LR) * 8;
          const int lm = wr0 + 16 * i + r;
          const int gc = n0 + wn * WC + c8;
          if (lm < m_valid && gc < p.N) {
            const float* sp = strip + r * kP + c8;
            if constexpr (MODE == M_DW) {
              float* dst = dw_dst(row0 + lm, gc);
              *reinterpret_cast<float4*>(dst) = make_float4(sp[0], sp[1], sp[2], sp[3]);
              *reinterpret_cast<float4*>(dst + 4) = make_float4(sp[4], sp[5], sp[6], sp[7]);
            } else {
              float v[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) v[e] = sp[e];
              const int64_t grow = row0 + lm;
              if constexpr (MODE == M_FWD1) {
                if constexpr (ACT == ACT_RELU) {
                  // ReLU commutes with the rounding to bf16 (round(max(h, 0)) =
                  // max(round(h), 0)), and ReLU layers keep A alone
#pragma unroll
                  for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e], 0.f);
                } else {
                  // H rounded to bf16 once: the packed bits are stored and
                  // their values feed the activation
                  const uint4 hb = pack8(v);
                  float hh[8];
                  unpack8(hb, hh);
#pragma unroll
                  for (int e = 0; e < 8; ++e) v[e] = act_f(hh[e], ACT);
                  if (p.H1)
                    *reinterpret_cast<uint4*>(p.H1 + grow * p.ldh + static_cast<int64_t>(gc) * ES) = hb;
                }
              }
              store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, v);
            }
          }
        }
      }
    }
    };
    if constexpr (MODE == M_FWD1 || MODE == M_BWD_DA) {
      if (p.act == ACT_RELU) epilogue(std::integral_constant<int, ACT_RELU>{});
      else epilogue(std::integral_constant<int, ACT_GELU>{});
    } else {
      epilogue(std::integral_constant<int, ACT_SWIGLU>{});
    }
    __syncthreads();   // strips are free before the next tile's loads
  }
}

// ---------------------------------------------------------------------------
// transposed weights
// ---------------------------------------------------------------------------
// Transposed copy of expert weights (bf16), so that dX reads them
// K-contiguous: dst[g][n][k] = src1[g][k][n] for k < K1 and src2[g][k - K1][n]
// for K1 <= k < K1 + K2 (dst rows of K1 + K2 elements).  A workgroup moves a
// 64 (k) x 64 (n) block through LDS: 16-byte loads along n, 16-byte stores
// along k.  K1, K2 and N are multiples of 8, so no vector straddles an edge
// or the seam between the two sources.
constexpr int kTr = 64;
__global__ __launch_bounds__(256) void transpose_w_kernel(const uint16_t* __restrict__ src1,
                                                          const uint16_t* __restrict__ src2,
                                                          int K1, int K2, int N,
                                                          uint16_t* __restrict__ dst) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[kTr][kTr + 8];
  const int g = blockIdx.z;
  const int n0 = blockIdx.x * kTr;
  const int K = K1 + K2;
  const int64_t s1 = static_cast<int64_t>(g) * K1 * N, s2 = static_cast<int64_t>(g) * K2 * N;
  for (int k0 = blockIdx.y * kTr; k0 < K; k0 += gridDim.y * kTr) {
    __syncthreads();   // the previous block's reads of the tile are done
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int kk = c >> 3, nn = (c & 7) * 8;
      const int k = k0 + kk, n = n0 + nn;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (k < K && n < N) {
        const uint16_t* src = k < K1 ? src1 + s1 + static_cast<int64_t>(k) * N + n
                                     : src2 + s2 + static_cast<int64_t>(k - K1) * N + n;
        v = *reinterpret_cast<const uint4*>(src);
      }
      *reinterpret_cast<uint4*>(&tile[kk][nn]) = v;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + 256 * i;
      const int nn = c >> 3, kk = (c & 7) * 8;
      const int n = n0 + nn, k = k0 + kk;
      if (n < N && k < K) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = static_cast<uint32_t>(tile[kk + 2 * j][nn]) |
                 (static_cast<uint32_t>(tile[kk + 2 * j + 1][nn]) << 16);
        *reinterpret_cast<uint4*>(dst + (static_cast<int64_t>(g) * N + n) * K + k) =
            make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// split-K reduction
// ---------------------------------------------------------------------------
// dW[g] = sum over the expert's split slots, in slot order.  A bounded grid
// strides over the elements (blockIdx.y = expert), so experts without a
// split cost one early exit per block rather than a launch per 1024
// elements.
constexpr int kReduceBlocks = 1024;   // blocks per expert

// The slots are added in slot order; their loads are issued four at a time
// ahead of the adds, so a thread waits out one memory latency per four slots.
__global__ __launch_bounds__(256) void split_reduce_kernel(
    const float* __restrict__ partial, int64_t slot_elems, const Sched* __restrict__ sc,
    float* __restrict__ dwA, float* __restrict__ dwB, int64_t dw_gstride, int split_row,
    int N) {
  const int g = blockIdx.y;
  const int ns = sc->nsplit[g];
  if (ns <= 1) return;
  const float* base = partial + static_cast<int64_t>(sc->slot0[g]) * slot_elems;
  auto add = [](float4& a, const float4& v) { a.x += v.x; a.y += v.y; a.z += v.z; a.w += v.w; };
  for (int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4; i < slot_elems;
       i += static_cast<int64_t>(gridDim.x) * 1024) {
    const float* p0 = base + i;
    float4 acc = *reinterpret_cast<const float4*>(p0);
    int sl = 1;
    for (; sl + 3 < ns; sl += 4) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        v[u] = *reinterpret_cast<const float4*>(p0 + static_cast<int64_t>(sl + u) * slot_elems);
#pragma unroll
      for (int u = 0; u < 4; ++u) add(acc, v[u]);
    }
    for (; sl < ns; ++sl) add(acc, *reinterpret_cast<const float4*>(p0 + static_cast<int64_t>(sl) * slot_elems));
    int64_t row, col;
    if (slot_elems < (int64_t(1) << 31)) {   // the usual case: 32-bit division
      const uint32_t ii = static_cast<uint32_t>(i);
      row = ii / static_cast<uint32_t>(N);
      col = ii % static_cast<uint32_t>(N);
    } else {
      row = i / N;
      col = i % N;
    }
    float* dst = row < split_row
                     ? dwA + static_cast<int64_t>(g) * dw_gstride + row * N + col
                     : dwB + static_cast<int64_t>(g) * dw_gstride + (row - split_row) * N + col;
    *reinterpret_cast<float4*>(dst) = acc;
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
int persistent_grid() {
  const int n = num_cus();
  return (n + kXcds - 1) / kXcds * kXcds;
}

inline int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// [rows_alloc, f] planes of h_save: A (ReLU), H and A (GELU), H1, H3 and A
// (SwiGLU).
int h_save_planes(moe_act act) { return act == MOE_SWIGLU ? 3 : act == MOE_GELU_TANH ? 2 : 1; }

// Sizes of the schedule and of every workspace buffer.
struct FfnPlan {
  int E, d, f, F;            // F = f (relu/gelu) or 2f (swiglu)
  int64_t rows_alloc;
  size_t es;
  int max_mtiles, max_mtiles_s, max_segs, max_slots, tmn_min;
  int64_t slot_elems;
  // byte offsets inside the workspace
  size_t o_sched, o_mtile, o_mtile_s, o_seg, o_end_sched;
  size_t o_abuf, o_dh, o_part, o_wt13, total_fwd, total_bwd, total_bwd_wt;
};

bool make_plan(moe_dtype dt, moe_act act, int E, int d, int f, int64_t rows_alloc, FfnPlan& pl) {
  if (!dtype_ok(dt) || E < 1 || E > kMaxE || !width_ok(d) || !width_ok(f) || !rows_ok(rows_alloc))
    return false;
  if (act != MOE_RELU && act != MOE_GELU_TANH && act != MOE_SWIGLU) return false;
  pl.E = E; pl.d = d; pl.f = f; pl.F = act == MOE_SWIGLU ? 2 * f : f;
  pl.rows_alloc = rows_alloc;
  pl.es = esize(dt);
  // every operand offset inside a 256-row tile (K-contiguous operands) or a
  // K step (K-major ones) stays below 2^31 bytes: buffer loads take 32-bit
  // offsets
  const int64_t max_ld = static_cast<int64_t>(pl.es) * (2 * static_cast<int64_t>(f) > d ? 2 * static_cast<int64_t>(f) : d);
  if (max_ld > kMaxOperandRowBytes) return false;
  pl.max_mtiles = cdiv(rows_alloc, BM) + E;
  pl.max_mtiles_s = cdiv(rows_alloc, BM_S) + E;
  const int tmn2 = cdiv(d, BM) * cdiv(f, BN);
  const int tmn13 = cdiv(pl.F, BM) * cdiv(d, BN);
  pl.tmn_min = tmn2 < tmn13 ? tmn2 : tmn13;
  const int64_t kcap = (rows_alloc + kKc - 1) / kKc * kKc + static_cast<int64_t>(kKc) * E;
  const int64_t slots_a = 1024 / pl.tmn_min;
  const int64_t slots_b = 2 * kcap / kSplitFloor;
  pl.max_slots = static_cast<int>(slots_a < slots_b ? slots_a : slots_b) + 1;
  pl.max_segs = E + pl.max_slots;
  pl.slot_elems = static_cast<int64_t>(pl.F) * d > static_cast<int64_t>(d) * f
                      ? static_cast<int64_t>(pl.F) * d : static_cast<int64_t>(d) * f;
  size_t o = 0;
  pl.o_sched = o; o = align_up(o + sizeof(Sched), 256);
  pl.o_mtile = o; o = align_up(o + sizeof(int2) * pl.max_mtiles, 256);
  pl.o_mtile_s = o; o = align_up(o + sizeof(int2) * pl.max_mtiles_s, 256);
  pl.o_seg = o;   o = align_up(o + sizeof(int4) * pl.max_segs, 256);
  pl.o_end_sched = o;
  const size_t es = pl.es;
  // forward: the activation buffer A [rows_alloc, f] when no h_save is given
  pl.o_abuf = o;
  pl.total_fwd = align_up(o + static_cast<size_t>(rows_alloc) * f * es, 256);
  // backward: dH [rows_alloc, F] and the split partial sums
  o = pl.o_end_sched;
  pl.o_dh = o;   o = align_up(o + static_cast<size_t>(rows_alloc) * pl.F * es, 256);
  pl.o_part = o; o = align_up(o + static_cast<size_t>(pl.max_slots) * pl.slot_elems * 4, 256);
  pl.total_bwd = o;
  // bf16: room for the transposed copy of [W1; W3] that dX may read
  // ([E, d, F]: row n of expert e = [W1_e[:, n]; W3_e[:, n]])
  pl.o_wt13 = o;
  pl.total_bwd_wt = dt == MOE_BF16 ? align_up(o + static_cast<size_t>(E) * d * pl.F * es, 256) : o;
  return true;
}

moe_status launch_schedule(hipStream_t s, const FfnPlan& pl, const int32_t* offsets,
                           const int32_t* rows, char* ws) {
  MOE_TIMED("ffn_schedule", s);
  schedule_kernel<<<1, 64, 0, s>>>(
      offsets, rows, pl.E, pl.rows_alloc, pl.max_mtiles, pl.max_mtiles_s, pl.max_segs, pl.tmn_min,
      pl.max_slots, reinterpret_cast<Sched*>(ws + pl.o_sched),
      reinterpret_cast<int2*>(ws + pl.o_mtile), reinterpret_cast<int2*>(ws + pl.o_mtile_s),
      reinterpret_cast<int4*>(ws + pl.o_seg));
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

GemmParams base_params(const FfnPlan& pl, const int32_t* offsets, char* ws) {
  GemmParams p{};
  p.offsets = offsets;
  p.sched = reinterpret_cast<const Sched*>(ws + pl.o_sched);
  p.mtile = reinterpret_cast<const int2*>(ws + pl.o_mtile);
  p.seg = reinterpret_cast<const int4*>(ws + pl.o_seg);
  p.kmsplit = 0x7FFFFFFF;
  return p;
}

// Tile choice of the bf16 products (moe_set_gemm_tiles: 0 automatic, 1 the
// 256x256 kernel only, 2 the 128x128 kernel only).
int g_tile_mode = 0;

// The 128x128 kernel runs two workgroups per CU, so one's prologue and
// epilogue overlap the other's MFMAs, but it reads twice the operand bytes
// per flop: on products that fill every CU for many rounds it takes about
// 1.3 times as long per flop as the 256x256 kernel.  It pays off where the
// 256x256 tiles leave CUs idle, mostly in the last round.  The host knows
// N, K and the row budget, not the per-expert rows, so it estimates both
// kernels' tile counts as if each expert held rows_alloc / E rows, counts
// the rounds of the persistent grids (one 256x256 tile or two 128x128
// tiles per CU at a time), and takes the 128x128 kernel when its rounds,
// each worth about 0.65 of a 256x256 round, take less time.  With K of 512
// or less (8 K steps per tile) a 256x256 tile's unoverlapped prologue and
// epilogue weigh more, and a 128x128 round is worth about 0.55 of one
// (measured on 512 x 2048 products of 1000-row experts).  K = 0: not known
// on the host (weight gradients).
bool use_small_tiles(const FfnPlan& pl, moe_dtype dt, bool vark, bool gated, int N, int M_out,
                     int K) {
  if (dt != MOE_BF16) return false;
  if (g_tile_mode == 1) return false;
  if (g_tile_mode == 2) return true;
  const int64_t per = cdiv(pl.rows_alloc, pl.E);
  auto tiles = [&](int tm, int tn) -> int64_t {
    const int64_t nt = cdiv(N, gated ? tn / 2 : tn);
    return vark ? static_cast<int64_t>(pl.E) * cdiv(M_out, tm) * nt
                : static_cast<int64_t>(pl.E) * cdiv(per, tm) * nt;
  };
  const int64_t G = persistent_grid();
  const int64_t rounds_big = (tiles(BM, BN) + G - 1) / G;
  const int64_t rounds_small = (tiles(BM_S, BM_S) + 2 * G - 1) / (2 * G);
  const int64_t w = K > 0 && K <= 512 ? 11 : 13;
  return w * rounds_small < 20 * rounds_big;
}

// dX with a transposed copy of [W1; W3] (moe_set_dx_weight_copy: 0
// automatic, 1 never, 2 always; bf16 only).  Read K-major, the weights need
// two transpose reads per MFMA fragment; read K-contiguous, dX ran 8-9%
// faster on 16384-row experts (same box, c5 and c4 shapes), and the copy
// moves 4 E d F bytes at about 5 TB/s.  The copy pays for itself from about
// 6000 rows per expert; the rule takes it from 8192 (rows_alloc / E: the
// row budget, as the host knows no fills).
int g_wt_mode = 0;
constexpr int64_t kWtRowsPerExpert = 8192;

bool use_wt13(const FfnPlan& pl, moe_dtype dt) {
  if (dt != MOE_BF16 || g_wt_mode == 1) return false;
  return g_wt_mode == 2 || pl.rows_alloc >= kWtRowsPerExpert * pl.E;
}

const char* pass_name(int pass) {
  static const char* names[] = {"gemm_fwd_h", "gemm_fwd_y", "gemm_bwd_da", "gemm_bwd_dx",
                                "gemm_bwd_dw2", "gemm_bwd_dw13", "gemm_bwd_dx"};
  return names[pass];
}

// Launches one product; sets the tile counts along N (and M for the weight
// gradients) for the kernel it picks.
template <int MODE, int PASS>
moe_status launch_gemm(hipStream_t s, moe_dtype dt, const FfnPlan& pl, char* ws, GemmParams p) {
  constexpr bool VARK = MODE == M_DW, GATED = MODE == M_FWD1_SWIGLU;
  const bool small = use_small_tiles(pl, dt, VARK, GATED, p.N, p.M_out, VARK ? 0 : p.K);
  const int tm = small ? BM_S : BM, tn = small ? BM_S : BN;
  p.ntiles = cdiv(p.N, GATED ? tn / 2 : tn);
  if (VARK) p.mtiles_out = cdiv(p.M_out, tm);
  if (small) p.mtile = reinterpret_cast<const int2*>(ws + pl.o_mtile_s);
  // the persistent grid, or fewer workgroups (a multiple of 8, for the XCD
  // mapping) when even the most tiles the schedule can list are fewer
  const int64_t max_items = VARK ? static_cast<int64_t>(pl.max_segs) * p.mtiles_out * p.ntiles
                                 : static_cast<int64_t>(small ? pl.max_mtiles_s : pl.max_mtiles) *
                                       p.ntiles;
  const int64_t full = (small ? 2 : 1) * static_cast<int64_t>(persistent_grid());
  const int grid = static_cast<int>(std::min(full, std::max<int64_t>(kXcds, (max_items + kXcds - 1) / kXcds * kXcds)));
  if constexpr ((MODE == M_FWD1 || MODE == M_FWD1_SWIGLU || MODE == M_STORE) &&
                (PASS == P_FWD_H || PASS == P_FWD_Y)) {
    // fp32 forward with few rows: one wavefront per 32x32 output block
    const int64_t mb = cdiv(pl.rows_alloc, kTinyB), nb = cdiv(p.N, kTinyB);
    const int64_t items = static_cast<int64_t>(pl.E) * mb * nb;
    if (dt == MOE_F32 && g_tile_mode != 1 && items <= kTinyMaxItems) {
      MOE_TIMED(pass_name(PASS), s);
      ffn_gemm_f32_tiny_kernel<MODE><<<static_cast<unsigned>(cdiv(items, 4)), 256, 0, s>>>(
          p, pl.E, static_cast<int>(mb), static_cast<int>(nb));
      MOE_LAUNCH_CHECK();
      return MOE_OK;
    }
  }
  MOE_TIMED(pass_name(PASS), s);
  if (dt == MOE_BF16 && small)
    ffn_gemm16_kernel<MODE, PASS, TileSmall><<<grid, kThreads16, 0, s>>>(p);
  else if (dt == MOE_BF16)
    ffn_gemm16_kernel<MODE, PASS, TileBig><<<grid, kThreads16, 0, s>>>(p);
  else
    ffn_gemm_f32_kernel<MODE, PASS><<<grid, kThreads, 0, s>>>(p);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

#define MOE_TRY(...)                       \
  do {                                     \
    moe_status st_ = (__VA_ARGS__);        \
    if (st_ != MOE_OK) return st_;         \
  } while (0)

// dW[g] = sum of expert g's split slots: rows [0, split_row) of the [M_out, N]
// result go to dwA, the rest to dwB; dw_gstride is the per-expert stride of
// dwA and dwB (f x d for [dW1; dW3], whose M_out is 2f under SwiGLU).
moe_status launch_split_reduce(hipStream_t s, const FfnPlan& pl, char* ws, int M_out, int N,
                               float* dwA, float* dwB, int split_row, int64_t dw_gstride) {
  const int64_t elems = static_cast<int64_t>(M_out) * N;
  const int64_t bx = cdiv(elems, 1024);
  dim3 grid(static_cast<unsigned>(bx < kReduceBlocks ? bx : kReduceBlocks), pl.E);
  MOE_TIMED("split_reduce", s);
  split_reduce_kernel<<<grid, 256, 0, s>>>(
      reinterpret_cast<const float*>(ws + pl.o_part), elems,
      reinterpret_cast<const Sched*>(ws + pl.o_sched), dwA, dwB, dw_gstride, split_row, N);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

// dst[g] = [src1[g]; src2[g]]^T for g < E (src1 [K1, N], src2 [K2, N] per expert).
moe_status launch_transpose_w(hipStream_t s, int E, const void* src1, const void* src2, int K1,
                              int K2, int N, void* dst) {
  const dim3 grid(cdiv(N, kTr), std::min(cdiv(K1 + K2, kTr), 32768), E);
  MOE_TIMED("transpose_w", s);
  transpose_w_kernel<<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(src1),
                                          static_cast<const uint16_t*>(src2), K1, K2, N,
                                          static_cast<uint16_t*>(dst));
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" moe_status moe_set_gemm_tiles(int mode) {
  if (mode < 0 || mode > 2) return MOE_EINVAL;
  g_tile_mode = mode;
  return MOE_OK;
}

extern "C" size_t moe_ffn_fwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d, int f,
                                              int64_t rows_alloc) {
  FfnPlan pl;
  return make_plan(dt, act, E, d, f, rows_alloc, pl) ? pl.total_fwd : 0;
}

extern "C" size_t moe_ffn_bwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d, int f,
                                              int64_t rows_alloc) {
  FfnPlan pl;
  if (!make_plan(dt, act, E, d, f, rows_alloc, pl)) return 0;
  return use_wt13(pl, dt) ? pl.total_bwd_wt : pl.total_bwd;
}

extern "C" moe_status moe_set_dx_weight_copy(int mode) {
  if (mode < 0 || mode > 2) return MOE_EINVAL;
  g_wt_mode = mode;
  return MOE_OK;
}

extern "C" moe_status moe_expert_ffn_fwd(void* stream, moe_dtype dt, moe_act act, int E, int d,
                                         int f, const int32_t* offsets, const int32_t* rows,
                                         int64_t rows_alloc, const void* x_disp, const void* w1,
                                         const void* w3, const void* w2, void* h_save,
                                         void* y_disp, void* workspace, size_t workspace_bytes) {
  FfnPlan pl;
  if (!make_plan(dt, act, E, d, f, rows_alloc, pl)) return MOE_EINVAL;
  if (!offsets || !rows || !w1 || !w2) return MOE_EINVAL;
  if (act == MOE_SWIGLU && !w3) return MOE_EINVAL;
  if (rows_alloc > 0 && (!x_disp || !y_disp)) return MOE_EINVAL;
  if (!aligned16(w1) || !aligned16(w2) || (w3 && !aligned16(w3)) ||
      (x_disp && !aligned16(x_disp)) || (y_disp && !aligned16(y_disp)) ||
      (h_save && !aligned16(h_save)))
    return MOE_EINVAL;
  if (rows_alloc == 0) return MOE_OK;
  if (!workspace || workspace_bytes < pl.total_fwd || !aligned16(workspace)) return MOE_EWORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  MOE_TRY(launch_schedule(s, pl, offsets, rows, ws));
  const int64_t es = static_cast<int64_t>(pl.es);
  const int64_t plane = rows_alloc * f * es;   // one [rows_alloc, f] plane of h_save
  const bool sw = act == MOE_SWIGLU;
  // A = act(H): the last plane of h_save when the caller keeps activations.
  // ReLU keeps A alone (relu'(H) = [A > 0]), so H is never written there.
  const int h_planes = h_save_planes(act) - 1;
  char* abuf = h_save ? static_cast<char*>(h_save) + h_planes * plane : ws + pl.o_abuf;

  GemmParams p = base_params(pl, offsets, ws);
  p.A = static_cast<const char*>(x_disp);
  p.lda = d * es;
  p.B = static_cast<const char*>(w1);
  p.B2 = static_cast<const char*>(w3);
  p.ldb = d * es;
  p.b_gstride = static_cast<int64_t>(f) * d * es;
  p.K = d;
  p.N = f;
  p.act = act == MOE_RELU ? ACT_RELU : (act == MOE_GELU_TANH ? ACT_GELU : ACT_SWIGLU);
  p.C = abuf;
  p.ldc = f * es;
  p.H1 = h_planes > 0 ? static_cast<char*>(h_save) : nullptr;
  p.H3 = h_save && sw ? static_cast<char*>(h_save) + plane : nullptr;
  p.ldh = f * es;
  if (sw) MOE_TRY(launch_gemm<M_FWD1_SWIGLU, P_FWD_H>(s, dt, pl, ws, p));
  else MOE_TRY(launch_gemm<M_FWD1, P_FWD_H>(s, dt, pl, ws, p));

  GemmParams q = base_params(pl, offsets, ws);
  q.A = abuf;
  q.lda = f * es;
  q.B = static_cast<const char*>(w2);
  q.ldb = f * es;
  q.b_gstride = static_cast<int64_t>(d) * f * es;
  q.K = f;
  q.N = d;
  q.C = static_cast<char*>(y_disp);
  q.ldc = d * es;
  MOE_TRY(launch_gemm<M_STORE, P_FWD_Y>(s, dt, pl, ws, q));
  return MOE_OK;
}

extern "C" moe_status moe_expert_ffn_bwd(void* stream, moe_dtype dt, moe_act act, int E, int d,
                                         int f, const int32_t* offsets, const int32_t* rows,
                                         int64_t rows_alloc, const void* x_disp,
                                         const void* h_save, const void* w1, const void* w3,
                                         const void* w2, const void* dy_disp, void* dx_disp,
                                         float* dw1, float* dw3, float* dw2, void* workspace,
                                         size_t workspace_bytes) {
  FfnPlan pl;
  if (!make_plan(dt, act, E, d, f, rows_alloc, pl)) return MOE_EINVAL;
  if (!offsets || !rows || !w1 || !w2 || !dw1 || !dw2) return MOE_EINVAL;
  if (act == MOE_SWIGLU && (!w3 || !dw3)) return MOE_EINVAL;
  if (rows_alloc > 0 && (!x_disp || !h_save || !dy_disp || !dx_disp)) return MOE_EINVAL;
  if (!aligned16(w1) || !aligned16(w2) || (w3 && !aligned16(w3)) || !aligned16(dw1) ||
      !aligned16(dw2) || (dw3 && !aligned16(dw3)) || (x_disp && !aligned16(x_disp)) ||
      (h_save && !aligned16(h_save)) || (dy_disp && !aligned16(dy_disp)) ||
      (dx_disp && !aligned16(dx_disp)))
    return MOE_EINVAL;
  if (!workspace || workspace_bytes < pl.total_bwd || !aligned16(workspace)) return MOE_EWORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  MOE_TRY(launch_schedule(s, pl, offsets, rows, ws));
  const int64_t es = static_cast<int64_t>(pl.es);
  const bool sw = act == MOE_SWIGLU;
  const int F = pl.F;
  char* dh = ws + pl.o_dh;      // [rows_alloc, F]: dH, or [dH1 | dH3]
  const int actc = act == MOE_RELU ? ACT_RELU : (act == MOE_GELU_TANH ? ACT_GELU : ACT_SWIGLU);
  const int64_t plane = rows_alloc * f * es;
  // A = act(H), saved by the forward after H (or H1, H3); ReLU saves A alone
  // and its derivative reads A: relu'(H) = [H > 0] = [A > 0]
  const char* abuf = static_cast<const char*>(h_save) + (h_save_planes(act) - 1) * plane;
  const char* h1 = act == MOE_RELU ? abuf : static_cast<const char*>(h_save);
  const char* h3 = sw ? h1 + plane : nullptr;

  // dX reads [W1; W3] from a transposed copy (K-contiguous) when the rule
  // or the caller's setting asks for it and the workspace has room for it
  const bool wt = use_wt13(pl, dt) && workspace_bytes >= pl.total_bwd_wt;
  char* wt13 = ws + pl.o_wt13;
  if (wt) MOE_TRY(launch_transpose_w(s, E, w1, sw ? w3 : nullptr, f, sw ? f : 0, d, wt13));

  // dx_disp = [dH1 | dH3] [W1; W3]: from the transposed copy, or W1, W3 read
  // K-major (W3 from k = f on)
  auto launch_dx = [&]() -> moe_status {
    if (wt) {
      GemmParams q = base_params(pl, offsets, ws);
      q.A = dh;
      q.lda = F * es;
      q.B = wt13;
      q.ldb = F * es;
      q.b_gstride = static_cast<int64_t>(d) * F * es;
      q.K = F;
      q.N = d;
      q.C = static_cast<char*>(dx_disp);
      q.ldc = d * es;
      return launch_gemm<M_STORE, P_BWD_DX_T>(s, dt, pl, ws, q);
    }
    GemmParams q = base_params(pl, offsets, ws);
    q.A = dh;
    q.lda = F * es;
    q.B = static_cast<const char*>(w1);
    q.B2 = sw ? static_cast<const char*>(w3) : nullptr;
    q.kmsplit = sw ? f : 0x7FFFFFFF;
    q.ldb = d * es;
    q.b_gstride = static_cast<int64_t>(f) * d * es;
    q.K = F;
    q.N = d;
    q.C = static_cast<char*>(dx_disp);
    q.ldc = d * es;
    return launch_gemm<M_STORE, P_BWD_DX>(s, dt, pl, ws, q);
  };
  // Order of the four products: dA first (it writes dH), dX right after it,
  // except when dx_disp is small enough to stay in the last-level cache: then
  // dX goes last, so the dispatch backward that follows reads dx_disp from
  // that cache rather than from HBM.
  const bool dx_last = rows_alloc * d * es <= kDxLastBytes;

  // dA = dY W2 (W2 read K-major: its rows are the d inputs) -> dH
  GemmParams p = base_params(pl, offsets, ws);
  p.A = static_cast<const char*>(dy_disp);
  p.lda = d * es;
  p.B = static_cast<const char*>(w2);
  p.ldb = f * es;
  p.b_gstride = static_cast<int64_t>(d) * f * es;
  p.K = d;
  p.N = f;
  p.act = actc;
  p.C = dh;
  p.ldc = F * es;
  p.H1 = const_cast<char*>(h1);
  p.H3 = const_cast<char*>(h3);
  p.ldh = f * es;
  p.f = f;
  if (sw) MOE_TRY(launch_gemm<M_BWD_DA_SWIGLU, P_BWD_DA>(s, dt, pl, ws, p));
  else MOE_TRY(launch_gemm<M_BWD_DA, P_BWD_DA>(s, dt, pl, ws, p));
  if (!dx_last) MOE_TRY(launch_dx());

  // dW2 [d, f] = dY^T A, contracting over each expert's dispatched rows
  GemmParams r = base_params(pl, offsets, ws);
  r.A = static_cast<const char*>(dy_disp);
  r.lda = d * es;
  r.M_out = d;
  r.B = abuf;
  r.ldb = f * es;
  r.N = f;
  r.dwA = dw2;
  r.dwB = dw2;
  r.dw_gstride = static_cast<int64_t>(d) * f;
  r.split_row = d;
  r.partial = reinterpret_cast<float*>(ws + pl.o_part);
  r.slot_elems = static_cast<int64_t>(d) * f;
  MOE_TRY(launch_gemm<M_DW, P_BWD_DW2>(s, dt, pl, ws, r));
  MOE_TRY(launch_split_reduce(s, pl, ws, d, f, dw2, dw2, d, r.dw_gstride));

  // [dW1; dW3] [F, d] = [dH1 dH3]^T X
  GemmParams u = base_params(pl, offsets, ws);
  u.A = dh;
  u.lda = F * es;
  u.M_out = F;
  u.B = static_cast<const char*>(x_disp);
  u.ldb = d * es;
  u.N = d;
  u.dwA = dw1;
  u.dwB = sw ? dw3 : dw1;
  u.dw_gstride = static_cast<int64_t>(f) * d;
  u.split_row = f;
  u.partial = reinterpret_cast<float*>(ws + pl.o_part);
  u.slot_elems = static_cast<int64_t>(F) * d;
  MOE_TRY(launch_gemm<M_DW, P_BWD_DW13>(s, dt, pl, ws, u));
  MOE_TRY(launch_split_reduce(s, pl, ws, F, d, dw1, sw ? dw3 : dw1, f, u.dw_gstride));

  // dx_disp last when it fits the last-level cache (see kDxLastBytes)
  if (dx_last) MOE_TRY(launch_dx());
  return MOE_OK;
}
