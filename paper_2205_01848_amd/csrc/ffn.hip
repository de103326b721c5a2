// Expert FFN of the MoE layer (the expert modules E_e of Algorithm 1) on
// dynamically sized per-expert tensors (Section 3.1), forward and backward.
//
// Every product is one persistent grouped GEMM kernel in "NT" form,
//     C[m, n] = sum_k A[m, k] * B[n, k]     (both operands K-contiguous),
// 256x256 output tiles, K tiles of 128 bytes, 8 wavefronts of 128x64 each
// on v_mfma_f32_32x32x16_bf16 (fp32 layers: v_mfma_f32_32x32x2f32) in two
// ping-pong teams (one team's MFMAs overlap the other's LDS reads), operand
// tiles loaded HBM -> LDS by buffer loads, double-buffered, with an XOR
// swizzle that keeps the MFMA fragment reads bank-conflict free.
//  * var-M products (forward H, Y; backward dA, dX): the M dimension of
//    expert e is its row count, read on the device; tiles are listed by a
//    one-workgroup schedule kernel, so no host synchronisation is needed.
//  * var-K products (dW): K of expert e is its row count; the K range is
//    split into chunks only when few experts carry most rows, and split
//    partial sums are added in a fixed order (deterministic).
// The persistent grid maps workgroup b to XCD b % 8 and hands each XCD a
// contiguous run of tiles arranged as 4 M-tiles x 8 N-tiles, so tiles that
// share operand panels share that XCD's L2.
// Epilogues (activation, SwiGLU, activation backward, transposed stores) run
// per wavefront on its fp32 accumulators, staged 16 rows at a time through a
// private LDS strip, and write 16-byte vectors.

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

constexpr int kGroupM = 4;      // M tiles per scheduling group
constexpr int kXcds = 8;
constexpr int kSplitFloor = 512;  // smallest K chunk of a split dW product
constexpr int kTT = 64;           // transpose tile
constexpr int64_t kMaxOperandRowBytes = (int64_t(1) << 23) - 64;  // 256 rows < 2^31 bytes

enum Act { ACT_RELU = 0, ACT_GELU = 1, ACT_SWIGLU = 2 };

// Device-side schedule written by schedule_kernel.
struct Sched {
  int n_mtiles;    // (expert, m0) tiles of BM rows
  int n_ttiles;    // (expert, r0) tiles of 64 rows for the transposes
  int n_segs;      // (expert, k range) segments of the dW products
  int kc;          // split chunk (rows)
  int kpad_total;  // columns used in the transposed buffers
  int n_slots;     // partial-sum slots used
  int pad_[2];
  int rows[kMaxE];    // clamped rows per expert
  int kbase[kMaxE];   // first column of expert e in the transposed buffers
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

// ---------------------------------------------------------------------------
// activations (shared by forward epilogue, backward epilogue and transposes)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float act_f(float h, int act) {
  if (act == ACT_RELU) return fmaxf(h, 0.f);
  // GELU, tanh form
  const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
  return 0.5f * h * (1.f + tanhf(u));
}
__device__ __forceinline__ float act_grad_f(float h, int act) {
  if (act == ACT_RELU) return h > 0.f ? 1.f : 0.f;
  const float u = 0.7978845608028654f * (h + 0.044715f * h * h * h);
  const float th = tanhf(u);
  const float du = 0.7978845608028654f * (1.f + 3.f * 0.044715f * h * h);
  return 0.5f * (1.f + th) + 0.5f * h * (1.f - th * th) * du;
}
__device__ __forceinline__ float sigm(float h) { return 1.f / (1.f + expf(-h)); }

// ---------------------------------------------------------------------------
// schedule
// ---------------------------------------------------------------------------
// One workgroup; thread 0 walks the experts in order.  Clamps every expert's
// rows to its region and to rows_alloc, and the totals to the host bounds
// the workspace was sized for, so no later kernel can index out of bounds.
__global__ void schedule_kernel(const int32_t* __restrict__ offsets,
                                const int32_t* __restrict__ rows, int E,
                                int64_t rows_alloc, int max_mtiles, int max_ttiles,
                                int kpad_cap, int max_segs, int tmn_min, int max_slots,
                                Sched* __restrict__ s, int2* __restrict__ mtile,
                                int2* __restrict__ ttile, int4* __restrict__ seg) {
  if (threadIdx.x != 0) return;
  int nm = 0, nt = 0, kb = 0;
  int64_t kwork = 0;
  for (int g = 0; g < E; ++g) {
    const int64_t off = offsets[g];
    int64_t m = rows[g];
    if (off < 0 || off >= rows_alloc) m = 0;
    m = min(m, static_cast<int64_t>(offsets[g + 1]) - off);
    m = min(m, rows_alloc - off);
    m = max(m, int64_t(0));
    // keep the tile lists and transposed columns inside their bounds
    const int64_t room_m = static_cast<int64_t>(max_mtiles - nm) * BM;
    const int64_t room_k = static_cast<int64_t>(kpad_cap - kb);
    m = min(m, room_m);
    m = min(m, room_k / kTT * kTT);
    m = min(m, static_cast<int64_t>(max_ttiles - nt) * kTT);
    const int mi = static_cast<int>(m);
    s->rows[g] = mi;
    for (int m0 = 0; m0 < mi; m0 += BM) mtile[nm++] = make_int2(g, m0);
    const int kp = (mi + kTT - 1) / kTT * kTT;
    s->kbase[g] = kb;
    for (int r0 = 0; r0 < kp; r0 += kTT) ttile[nt++] = make_int2(g, r0);
    kb += kp;
    kwork += kp;
  }
  s->n_mtiles = nm;
  s->n_ttiles = nt;
  s->kpad_total = kb;
  // K chunk: aim at about 2 x 256 work items over all split products
  int64_t kc = (kwork * tmn_min + 511) / 512;
  kc = (kc + kTT - 1) / kTT * kTT;
  kc = max(kc, static_cast<int64_t>(kSplitFloor));
  int ns = 0, slots = 0;
  for (int g = 0; g < E; ++g) {
    const int kp = (s->rows[g] + kTT - 1) / kTT * kTT;
    int nsp = kp > kc ? static_cast<int>((kp + kc - 1) / kc) : 1;
    if (nsp > 1 && (slots + nsp > max_slots || ns + nsp > max_segs)) nsp = 1;
    if (ns + nsp > max_segs) nsp = 0;  // cannot happen with host bounds; stay in bounds
    s->nsplit[g] = nsp;
    s->slot0[g] = nsp > 1 ? slots : -1;
    for (int i = 0; i < nsp; ++i) {
      const int k0 = static_cast<int>(min(static_cast<int64_t>(i) * kc, static_cast<int64_t>(kp)));
      const int k1 = static_cast<int>(min(static_cast<int64_t>(i + 1) * kc, static_cast<int64_t>(kp)));
      seg[ns++] = make_int4(g, nsp > 1 ? k0 : 0, nsp > 1 ? k1 : kp, nsp > 1 ? slots + i : -1);
    }
    if (nsp > 1) slots += nsp;
  }
  s->n_segs = ns;
  s->n_slots = slots;
  s->kc = static_cast<int>(kc);
}

// ---------------------------------------------------------------------------
// GEMM core
// ---------------------------------------------------------------------------
template <typename T> struct Mma;
template <> struct Mma<uint16_t> {
  __device__ static __forceinline__ void run(floatx16& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  __device__ static __forceinline__ void run(floatx16& c, const uint4& a, const uint4& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
};

// One tile's operand description (byte pointers, byte strides).  Rows of a
// tile at or past a_rows / b_rows, and K bytes at or past kbytes, read as 0.
struct TileOps {
  const char* a;      // A tile: row 0, k = 0
  int64_t lda;        // bytes between A rows
  int a_rows;         // valid A rows
  const char* b;      // B tile: row 0, k = 0
  const char* b3;     // gated forward: the W3 rows (b holds W1), else null
  int64_t ldb;
  int b_rows;         // valid B rows (gated forward: valid hidden units)
  int kbytes;         // K extent in bytes (multiple of 16)
};

// LDS tile layout: row r (0..255) of 128 bytes, its 16-byte chunk c stored at
// r*128 + ((c ^ ((r >> 1) & 7)) << 4).  gfx950 LDS serves 16 lanes of a
// 16-byte access per cycle from 64 banks (256 bytes): the MFMA fragment reads
// touch 16 consecutive rows at one logical chunk; rows alternate bank halves
// and (r >> 1) & 7 spreads each half's 8 rows over its 8 slots.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

// Buffer resource over a tile's operand.  Every offset used is below 2^31
// (host limits), so 0x80000000 is always out of range: a lane given that
// offset loads zeros, which is how ragged rows and K tails are filled.
constexpr uint32_t kOob = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const char* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), static_cast<short>(0),
                                           0x7FFFFFFF, 0x00020000);
}
#define MOE_LDS(p) ((__attribute__((address_space(3))) void*)(p))

// acc += A_tile * B_tile^T over the whole K extent: 8 wavefronts in two
// teams of four, one wave of each team per SIMD.  Team t computes tile rows
// 128t..128t+127, its wave q columns 64q..64q+63 (gated forward: hidden units
// 32q..32q+31, W1 then W3).  Each half K step (32 bf16) is a memory phase
// (12 fragment reads, LDS -> registers) followed by an MFMA phase (16 MFMAs
// from registers).  Team 1 runs one barrier behind team 0, so while one wave
// of a SIMD issues MFMAs the other reads LDS.  Operand tiles go HBM -> LDS
// with buffer_load ... lds (no register staging), issued by team 0 one step
// ahead into the other of two stages.
template <typename T, bool GATED, bool FULL>
__device__ __forceinline__ void mainloop(const TileOps& op, char* la0, char* lb0, char* la1,
                                         char* lb1, floatx16 (&acc)[4][2]) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int team = wave >> 2, wq = wave & 3;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  const int kbytes = op.kbytes;
  const int nk = (kbytes + kRowBytes - 1) / kRowBytes;
  if (nk <= 0) return;
  const int nk2 = (nk + 1) & ~1;   // odd counts load one all-zero step

  // Loads: 8-row block blk of an operand, lane l -> tile row blk*8 + (l >> 3),
  // physical chunk l & 7, logical chunk (l & 7) ^ swz(row), which depends on
  // the parity of blk only.
  const int l3 = lane >> 3;
  const int co0 = ((lane & 7) ^ swz(l3)) * 16, co1 = ((lane & 7) ^ swz(l3 + 8)) * 16;
  const uint32_t la_row = static_cast<uint32_t>(l3 * op.lda);
  const uint32_t lb_row = static_cast<uint32_t>(l3 * op.ldb);
  const __amdgpu_buffer_rsrc_t ra = tile_rsrc(op.a);
  const __amdgpu_buffer_rsrc_t rb = tile_rsrc(op.b);
  const __amdgpu_buffer_rsrc_t rb3 = tile_rsrc(GATED ? op.b3 : op.b);
  const int lda = static_cast<int>(op.lda), ldb = static_cast<int>(op.ldb);
  // FULL: every row valid and K a whole number of steps, so a step is either
  // entirely inside K or (the padding step) entirely outside.  Otherwise
  // each lane checks its row and its K chunk.
  auto load = [&](int kt, char* sa, char* sb, int b0, int nb) {
    const int kofs = kt * kRowBytes;
    const bool kin = kofs < kbytes;   // wave-uniform
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i < nb) {
        const int blk = b0 + i;
        const int co = (i & 1) ? co1 : co0;   // b0 is even
        // B row of this block: plain, or W1/W3 groups of 32 (gated forward)
        const int brow0 = GATED ? (blk >> 3) * 32 + (blk & 3) * 8 : blk * 8;
        uint32_t oa = la_row + co, ob = lb_row + co;
        if constexpr (FULL) {
          if (!kin) oa = ob = kOob;
        } else {
          const bool kok = kofs + co < kbytes;
          if (!kok || blk * 8 + l3 >= op.a_rows) oa = kOob;
          if (!kok || brow0 + l3 >= op.b_rows) ob = kOob;
        }
        const int sa_off = blk * 8 * lda + kofs;
        const int sb_off = brow0 * ldb + kofs;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, MOE_LDS(sa + blk * 1024), 16, oa, sa_off, 0, 0);
        if (GATED && ((blk >> 2) & 1))
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rb3, MOE_LDS(sb + blk * 1024), 16, ob, sb_off, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, MOE_LDS(sb + blk * 1024), 16, ob, sb_off, 0, 0);
      }
    }
  };

  const int fr_row = lane & 31;
  const int fr_a = (team * 128 + fr_row) * kRowBytes;
  const int fr_b = (wq * 64 + fr_row) * kRowBytes;
  uint4 fa[4][2], fb[2][2];   // [sub-tile][k sub-step within the half step]
  // fragments of k sub-steps 2h and 2h+1 (one half of a K step)
  auto fread = [&](const char* sa, const char* sb, int h) {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int sw = ((4 * h + 2 * s2 + (lane >> 5)) ^ swz(fr_row)) << 4;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        fa[i][s2] = *reinterpret_cast<const uint4*>(sa + fr_a + i * 32 * kRowBytes + sw);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        fb[j][s2] = *reinterpret_cast<const uint4*>(sb + fr_b + j * 32 * kRowBytes + sw);
    }
  };
  auto mma = [&]() {
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) Mma<T>::run(acc[i][j], fa[i][s2], fb[j][s2]);
  };
  // s_waitcnt immediates (gfx9 encoding)
  constexpr int kWaitVm0 = 0x0F70;    // vmcnt(0)
  constexpr int kWaitLgkm0 = 0xC07F;  // lgkmcnt(0)
  // one ping-pong phase pair: read half h of a stage, then its 16 MFMAs
  auto half = [&](const char* sa, const char* sb, int h, bool wait_loads) {
    fread(sa, sb, h);
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    mma();
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
  M_BWD_DA = 3,      // dA = dY W2 -> dH = dA act'(H), row-major + transposed
  M_BWD_DA_SWIGLU = 4,
  M_DW = 5           // var-K weight gradient, fp32
};

struct GemmParams {
  // operands (bytes)
  const char* A; int64_t lda;
  const char* B; const char* B2; int64_t ldb; int64_t b_gstride;
  int64_t kbytes;     // var-M: K extent in bytes
  int N;              // var-M: output columns;  var-K: output columns (N_out)
  int M_out;          // var-K: output rows
  int ntiles;         // tiles along N
  int mtiles_out;     // var-K: tiles along M
  int act;
  // outputs
  char* C; int64_t ldc;           // row-major output (bytes per row)
  char* H1; char* H3; int64_t ldh; // saved / read pre-activations (bytes per row)
  char* CT; int64_t ldct;          // transposed output (bytes per row)
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

// PASS only names the instance (forward H, forward Y, backward dA, dX, dW2,
// dW1/dW3), so each product is a separate kernel in traces.
enum Pass { P_FWD_H = 0, P_FWD_Y = 1, P_BWD_DA = 2, P_BWD_DX = 3, P_BWD_DW2 = 4, P_BWD_DW13 = 5 };

template <typename T, int MODE, int PASS>
__global__ __launch_bounds__(kThreads, 1) void ffn_gemm_kernel(const GemmParams p) {
  // two stages of the A and B tiles, four distinct objects (see mainloop);
  // after the K loop the same memory holds each wave's epilogue strips
  __shared__ __attribute__((aligned(16))) char la0[kTileBytes];
  __shared__ __attribute__((aligned(16))) char lb0[kTileBytes];
  __shared__ __attribute__((aligned(16))) char la1[kTileBytes];
  __shared__ __attribute__((aligned(16))) char lb1[kTileBytes];
  constexpr int ES = sizeof(T);
  constexpr bool VARK = MODE == M_DW;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int team = wave >> 2, wq = wave & 3;
  const Sched& sc = *p.sched;
  const int n_items = VARK ? sc.n_segs * p.mtiles_out * p.ntiles : sc.n_mtiles * p.ntiles;
  const int G = gridDim.x;
  const int lbase = (blockIdx.x % kXcds) * (G / kXcds) + blockIdx.x / kXcds;
  // the wave's two staging strips (kStripsPerArray per 32 KB array)
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
    float* strip3 = strip_at(2 * wave + 1) + z;
    TileOps op;
    int g, row0, m_valid;       // var-M: expert, first global row, valid rows in tile
    int n0;                      // first output column of the tile
    int local_m0 = 0;            // var-M: first expert-local row
    int slot = -1, mt, nt;
    op.b3 = nullptr;
    if constexpr (!VARK) {
      int mti;
      decode_grouped(L, sc.n_mtiles, p.ntiles, mti, nt);
      const int2 tm = p.mtile[mti];
      g = tm.x;
      local_m0 = tm.y;
      row0 = p.offsets[g] + tm.y;
      m_valid = min(BM, sc.rows[g] - tm.y);
      op.a = p.A + static_cast<int64_t>(row0) * p.lda;
      op.lda = p.lda;
      op.a_rows = m_valid;
      op.kbytes = static_cast<int>(p.kbytes);
      op.ldb = p.ldb;
      const char* bg = p.B + static_cast<int64_t>(g) * p.b_gstride;
      if constexpr (MODE == M_FWD1_SWIGLU) {
        n0 = nt * (BN / 2);  // hidden units covered by this tile (W1 and W3 rows)
        op.b = bg + static_cast<int64_t>(n0) * p.ldb;
        op.b3 = p.B2 + static_cast<int64_t>(g) * p.b_gstride + static_cast<int64_t>(n0) * p.ldb;
        op.b_rows = min(BN / 2, p.N - n0);
      } else {
        n0 = nt * BN;
        op.b = bg + static_cast<int64_t>(n0) * p.ldb;
        op.b_rows = min(BN, p.N - n0);
      }
    } else {
      const int tmn = p.mtiles_out * p.ntiles;
      const int si = L / tmn;
      decode_grouped(L - si * tmn, p.mtiles_out, p.ntiles, mt, nt);
      const int4 sg = p.seg[si];
      g = sg.x;
      slot = sg.w;
      const int col = sc.kbase[g] + sg.y;   // first K column of this segment
      row0 = mt * BM;
      n0 = nt * BN;
      m_valid = min(BM, p.M_out - row0);
      op.a = p.A + static_cast<int64_t>(row0) * p.lda + static_cast<int64_t>(col) * ES;
      op.lda = p.lda;
      op.a_rows = m_valid;
      op.ldb = p.ldb;
      op.b = p.B + static_cast<int64_t>(n0) * p.ldb + static_cast<int64_t>(col) * ES;
      op.b_rows = min(BN, p.N - n0);
      op.kbytes = (sg.z - sg.y) * ES;
    }

    floatx16 acc[4][2];
    constexpr bool GATED = MODE == M_FWD1_SWIGLU;
    if (op.a_rows >= BM && op.b_rows >= (GATED ? BN / 2 : BN) && op.kbytes % kRowBytes == 0)
      mainloop<T, GATED, true>(op, la0, lb0, la1, lb1, acc);
    else
      mainloop<T, GATED, false>(op, la0, lb0, la1, lb1, acc);

    // Epilogue, wave by wave: 16 accumulator rows at a time go through the
    // wave's own LDS strip, then each lane finishes 8 consecutive columns of
    // a row and writes them as one vector.
    const int wcol = wq * 64;   // the wave's first tile column
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
        } else if constexpr (MODE == M_BWD_DA || MODE == M_BWD_DA_SWIGLU) {
          constexpr bool SW = MODE == M_BWD_DA_SWIGLU;
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const int r = it * 8 + (lane >> 3), c8 = (lane & 7) * 8;
            const int lm = srow0 + r;
            const int gc = n0 + wcol + c8;
            float g1[8], g3[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) g1[e] = g3[e] = 0.f;
            if (lm < m_valid && gc < p.N) {
              const int64_t grow = row0 + lm;
              float h1[8];
              load_vec<T>(p.H1 + grow * p.ldh + static_cast<int64_t>(gc) * ES, h1);
              if constexpr (SW) {
                float h3[8];
                load_vec<T>(p.H3 + grow * p.ldh + static_cast<int64_t>(gc) * ES, h3);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  const float da = strip[r * kStripPitch + c8 + e];
                  const float sg = sigm(h1[e]);
                  g1[e] = Elem<T>::to_f(Elem<T>::from_f(da * h3[e] * sg * (1.f + h1[e] * (1.f - sg))));
                  g3[e] = Elem<T>::to_f(Elem<T>::from_f(da * h1[e] * sg));
                }
                store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
                store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(p.f + gc) * ES, g3);
              } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                  g1[e] = Elem<T>::to_f(Elem<T>::from_f(strip[r * kStripPitch + c8 + e] *
                                                         act_grad_f(h1[e], p.act)));
                store_vec<T>(p.C + grow * p.ldc + static_cast<int64_t>(gc) * ES, g1);
              }
            }
            // keep the rounded gradients for the transposed store (in place:
            // each lane rewrites exactly the elements it read); rows past the
            // expert's rows become zero (the transposed buffers are zero-padded)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              strip[r * kStripPitch + c8 + e] = g1[e];
              if constexpr (SW) strip3[r * kStripPitch + c8 + e] = g3[e];
            }
          }
          // transposed store: 8 consecutive expert rows of one column per lane
          const int kcol0 = sc.kbase[g] + local_m0 + srow0;   // first transposed column
          const int kpad_g = (sc.rows[g] + kTT - 1) / kTT * kTT;
          const int gc = n0 + wcol + lane;
#pragma unroll
          for (int it = 0; it < 2; ++it) {
            const int rg = it * 8;
            if (gc < p.N && local_m0 + srow0 + rg < kpad_g) {
              float v[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) v[e] = strip[(rg + e) * kStripPitch + lane];
              store_vec<T>(p.CT + static_cast<int64_t>(gc) * p.ldct +
                               static_cast<int64_t>(kcol0 + rg) * ES, v);
              if constexpr (SW) {
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = strip3[(rg + e) * kStripPitch + lane];
                store_vec<T>(p.CT + static_cast<int64_t>(p.f + gc) * p.ldct +
                                 static_cast<int64_t>(kcol0 + rg) * ES, v);
              }
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
    __syncthreads();   // strips are free before the next tile's loads
  }
}

// ---------------------------------------------------------------------------
// transposes
// ---------------------------------------------------------------------------
enum TMode { T_COPY = 0, T_ACT = 1, T_SWIGLU = 2 };

// out[c, kbase[g] + r] = op(in[offsets[g] + r, c]) for the 64-row tile list,
// rows past the expert's rows (up to the 64 padding) written as zero.
template <typename T, int TM>
__global__ __launch_bounds__(256) void rows_transpose_kernel(
    const char* __restrict__ in, const char* __restrict__ in3, int64_t ld_in, int D,
    int act, const int32_t* __restrict__ offsets, const Sched* __restrict__ sc,
    const int2* __restrict__ ttile, char* __restrict__ out, int64_t ld_out) {
  constexpr int ES = sizeof(T);
  constexpr int V = 16 / ES;          // elements per 16-byte chunk
  constexpr int CPR = kTT / V;        // chunks per 64-element row
  __shared__ float tile[kTT][kTT + 1];
  if (static_cast<int>(blockIdx.x) >= sc->n_ttiles) return;
  const int2 tt = ttile[blockIdx.x];
  const int g = tt.x, r0 = tt.y;
  const int c0 = blockIdx.y * kTT;
  const int rows_g = sc->rows[g];
  const int64_t grow0 = static_cast<int64_t>(offsets[g]) + r0;
  for (int ch = threadIdx.x; ch < kTT * CPR; ch += 256) {
    const int rr = ch / CPR, cc = ch % CPR;
    const int col = c0 + cc * V;
    float v[V];
    if (r0 + rr < rows_g && col < D) {
      const int64_t o = (grow0 + rr) * ld_in + static_cast<int64_t>(col) * ES;
      const uint4 raw = *reinterpret_cast<const uint4*>(in + o);
      Elem<T>::load(raw, v);
      if constexpr (TM == T_ACT) {
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = act_f(v[e], act);
      } else if constexpr (TM == T_SWIGLU) {
        float h3[V];
        Elem<T>::load(*reinterpret_cast<const uint4*>(in3 + o), h3);
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = v[e] * sigm(v[e]) * h3[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) v[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < V; ++e) tile[rr][cc * V + e] = v[e];
  }
  __syncthreads();
  const int64_t kcol = static_cast<int64_t>(sc->kbase[g]) + r0;
  for (int ch = threadIdx.x; ch < kTT * CPR; ch += 256) {
    const int oc = ch / CPR, rc = ch % CPR;
    if (c0 + oc >= D) continue;
    float v[V];
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = tile[rc * V + e][oc];
    *reinterpret_cast<uint4*>(out + static_cast<int64_t>(c0 + oc) * ld_out +
                              (kcol + rc * V) * ES) = Elem<T>::store(v);
  }
}

// out[g, c, co + r] = in[g, r, c] for in [E, R, C] (weights), for the experts
// that have rows (the others' transposed weights are never read).
template <typename T>
__global__ __launch_bounds__(256) void weight_transpose_kernel(
    const T* __restrict__ in, int R, int C, T* __restrict__ out, int64_t ld_out, int co,
    int64_t out_gstride, const Sched* __restrict__ sc) {
  __shared__ T tile[kTT][kTT + 1];
  const int g = blockIdx.z;
  if (sc->rows[g] == 0) return;
  const int c0 = blockIdx.x * kTT, r0 = blockIdx.y * kTT;
  const T* src = in + static_cast<int64_t>(g) * R * C;
  T* dst = out + static_cast<int64_t>(g) * out_gstride;
  for (int i = threadIdx.x; i < kTT * kTT; i += 256) {
    const int rr = i / kTT, cc = i % kTT;
    if (r0 + rr < R && c0 + cc < C) tile[rr][cc] = src[static_cast<int64_t>(r0 + rr) * C + c0 + cc];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kTT * kTT; i += 256) {
    const int cc = i / kTT, rr = i % kTT;
    if (r0 + rr < R && c0 + cc < C)
      dst[static_cast<int64_t>(c0 + cc) * ld_out + co + r0 + rr] = tile[rr][cc];
  }
}

// dW[g] = sum over the expert's split slots, in slot order.
__global__ __launch_bounds__(256) void split_reduce_kernel(
    const float* __restrict__ partial, int64_t slot_elems, const Sched* __restrict__ sc,
    float* __restrict__ dwA, float* __restrict__ dwB, int64_t dw_gstride, int split_row,
    int N) {
  const int g = blockIdx.y;
  const int ns = sc->nsplit[g];
  if (ns <= 1) return;
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i >= slot_elems) return;
  const float* p0 = partial + static_cast<int64_t>(sc->slot0[g]) * slot_elems + i;
  float4 acc = *reinterpret_cast<const float4*>(p0);
  for (int s = 1; s < ns; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(p0 + static_cast<int64_t>(s) * slot_elems);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  const int64_t row = i / N, col = i % N;
  float* dst = row < split_row
                   ? dwA + static_cast<int64_t>(g) * dw_gstride + row * N + col
                   : dwB + static_cast<int64_t>(g) * dw_gstride + (row - split_row) * N + col;
  *reinterpret_cast<float4*>(dst) = acc;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
int num_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

int persistent_grid() {
  const int n = num_cus();
  return (n + kXcds - 1) / kXcds * kXcds;
}

inline int cdiv(int64_t a, int64_t b) { return static_cast<int>((a + b - 1) / b); }

// Sizes of the schedule and of every workspace buffer.
struct FfnPlan {
  int E, d, f, F;            // F = f (relu/gelu) or 2f (swiglu)
  int64_t rows_alloc;
  size_t es;
  int max_mtiles, max_ttiles, kpad_cap, max_segs, max_slots, tmn_min;
  int64_t slot_elems;
  // byte offsets inside the workspace
  size_t o_sched, o_mtile, o_ttile, o_seg, o_end_sched;
  size_t o_abuf, o_w2t, o_w13t, o_dh, o_dht, o_xt, o_dyt, o_at, o_part, total_fwd, total_bwd;
};

bool make_plan(moe_dtype dt, moe_act act, int E, int d, int f, int64_t rows_alloc, FfnPlan& pl) {
  if (!dtype_ok(dt) || E < 1 || E > kMaxE || !width_ok(d) || !width_ok(f) || !rows_ok(rows_alloc))
    return false;
  if (act != MOE_RELU && act != MOE_GELU_TANH && act != MOE_SWIGLU) return false;
  pl.E = E; pl.d = d; pl.f = f; pl.F = act == MOE_SWIGLU ? 2 * f : f;
  pl.rows_alloc = rows_alloc;
  pl.es = esize(dt);
  pl.max_mtiles = cdiv(rows_alloc, BM) + E;
  pl.max_ttiles = cdiv(rows_alloc, kTT) + E;
  const int64_t kcap = (rows_alloc + kTT - 1) / kTT * kTT + static_cast<int64_t>(kTT) * E;
  // every GEMM operand offset inside a 256-row tile stays below 2^31 bytes
  // (buffer-resource loads with 32-bit offsets)
  int64_t max_ld = kcap;
  if (2 * static_cast<int64_t>(f) > max_ld) max_ld = 2 * static_cast<int64_t>(f);
  if (d > max_ld) max_ld = d;
  if (max_ld * static_cast<int64_t>(pl.es) > kMaxOperandRowBytes) return false;
  pl.kpad_cap = static_cast<int>(kcap);
  const int tmn2 = cdiv(d, BM) * cdiv(f, BN);
  const int tmn13 = cdiv(pl.F, BM) * cdiv(d, BN);
  pl.tmn_min = tmn2 < tmn13 ? tmn2 : tmn13;
  int slots_a = 1024 / pl.tmn_min;
  int slots_b = static_cast<int>(2 * kcap / kSplitFloor);
  pl.max_slots = (slots_a < slots_b ? slots_a : slots_b) + 1;
  pl.max_segs = E + pl.max_slots;
  pl.slot_elems = static_cast<int64_t>(pl.F) * d > static_cast<int64_t>(d) * f
                      ? static_cast<int64_t>(pl.F) * d : static_cast<int64_t>(d) * f;
  size_t o = 0;
  pl.o_sched = o; o = align_up(o + sizeof(Sched), 256);
  pl.o_mtile = o; o = align_up(o + sizeof(int2) * pl.max_mtiles, 256);
  pl.o_ttile = o; o = align_up(o + sizeof(int2) * pl.max_ttiles, 256);
  pl.o_seg = o;   o = align_up(o + sizeof(int4) * pl.max_segs, 256);
  pl.o_end_sched = o;
  const size_t es = pl.es;
  // forward: the activation buffer A [rows_alloc, f]
  pl.o_abuf = o;
  pl.total_fwd = align_up(o + static_cast<size_t>(rows_alloc) * f * es, 256);
  // backward
  o = pl.o_end_sched;
  pl.o_w2t = o;  o = align_up(o + static_cast<size_t>(E) * f * d * es, 256);
  pl.o_w13t = o; o = align_up(o + static_cast<size_t>(E) * d * pl.F * es, 256);
  pl.o_dh = o;   o = align_up(o + static_cast<size_t>(rows_alloc) * pl.F * es, 256);
  pl.o_dht = o;  o = align_up(o + static_cast<size_t>(pl.F) * kcap * es, 256);
  pl.o_xt = o;   o = align_up(o + static_cast<size_t>(d) * kcap * es, 256);
  pl.o_dyt = o;  o = align_up(o + static_cast<size_t>(d) * kcap * es, 256);
  pl.o_at = o;   o = align_up(o + static_cast<size_t>(f) * kcap * es, 256);
  pl.o_part = o; o = align_up(o + static_cast<size_t>(pl.max_slots) * pl.slot_elems * 4, 256);
  pl.total_bwd = o;
  return true;
}

moe_status launch_schedule(hipStream_t s, const FfnPlan& pl, const int32_t* offsets,
                           const int32_t* rows, char* ws) {
  MOE_TIMED("ffn_schedule", s);
  schedule_kernel<<<1, 64, 0, s>>>(
      offsets, rows, pl.E, pl.rows_alloc, pl.max_mtiles, pl.max_ttiles, pl.kpad_cap,
      pl.max_segs, pl.tmn_min, pl.max_slots, reinterpret_cast<Sched*>(ws + pl.o_sched),
      reinterpret_cast<int2*>(ws + pl.o_mtile), reinterpret_cast<int2*>(ws + pl.o_ttile),
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
  return p;
}

const char* pass_name(int pass) {
  static const char* names[] = {"gemm_fwd_h", "gemm_fwd_y", "gemm_bwd_da", "gemm_bwd_dx",
                                "gemm_bwd_dw2", "gemm_bwd_dw13"};
  return names[pass];
}

template <int MODE, int PASS>
moe_status launch_gemm(hipStream_t s, moe_dtype dt, const GemmParams& p) {
  const int grid = persistent_grid();
  MOE_TIMED(pass_name(PASS), s);
  if (dt == MOE_BF16)
    ffn_gemm_kernel<uint16_t, MODE, PASS><<<grid, kThreads, 0, s>>>(p);
  else
    ffn_gemm_kernel<float, MODE, PASS><<<grid, kThreads, 0, s>>>(p);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

#define MOE_TRY(...)                       \
  do {                                     \
    moe_status st_ = (__VA_ARGS__);        \
    if (st_ != MOE_OK) return st_;         \
  } while (0)

template <int TM>
moe_status launch_rows_transpose(hipStream_t s, moe_dtype dt, const FfnPlan& pl,
                                 const int32_t* offsets, char* ws, const void* in,
                                 const void* in3, int D, int act, char* out) {
  dim3 grid(pl.max_ttiles, cdiv(D, kTT));
  const Sched* sc = reinterpret_cast<const Sched*>(ws + pl.o_sched);
  const int2* tt = reinterpret_cast<const int2*>(ws + pl.o_ttile);
  const int64_t ld_in = static_cast<int64_t>(D) * pl.es;
  const int64_t ld_out = static_cast<int64_t>(pl.kpad_cap) * pl.es;
  MOE_TIMED("transpose_rows", s);
  if (dt == MOE_BF16)
    rows_transpose_kernel<uint16_t, TM><<<grid, 256, 0, s>>>(
        static_cast<const char*>(in), static_cast<const char*>(in3), ld_in, D, act, offsets, sc,
        tt, out, ld_out);
  else
    rows_transpose_kernel<float, TM><<<grid, 256, 0, s>>>(
        static_cast<const char*>(in), static_cast<const char*>(in3), ld_in, D, act, offsets, sc,
        tt, out, ld_out);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

moe_status launch_weight_transpose(hipStream_t s, moe_dtype dt, const FfnPlan& pl, char* ws,
                                   const void* in, int E, int R, int C, char* out,
                                   int64_t ld_out, int co, int64_t gstride) {
  dim3 grid(cdiv(C, kTT), cdiv(R, kTT), E);
  const Sched* sc = reinterpret_cast<const Sched*>(ws + pl.o_sched);
  MOE_TIMED("transpose_weights", s);
  if (dt == MOE_BF16)
    weight_transpose_kernel<uint16_t><<<grid, 256, 0, s>>>(
        static_cast<const uint16_t*>(in), R, C, reinterpret_cast<uint16_t*>(out), ld_out, co,
        gstride, sc);
  else
    weight_transpose_kernel<float><<<grid, 256, 0, s>>>(
        static_cast<const float*>(in), R, C, reinterpret_cast<float*>(out), ld_out, co, gstride,
        sc);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

moe_status launch_split_reduce(hipStream_t s, const FfnPlan& pl, char* ws, int M_out, int N,
                               float* dwA, float* dwB, int split_row) {
  const int64_t elems = static_cast<int64_t>(M_out) * N;
  dim3 grid(cdiv(elems, 1024), pl.E);
  MOE_TIMED("split_reduce", s);
  split_reduce_kernel<<<grid, 256, 0, s>>>(
      reinterpret_cast<const float*>(ws + pl.o_part), elems,
      reinterpret_cast<const Sched*>(ws + pl.o_sched), dwA, dwB, static_cast<int64_t>(M_out) * N,
      split_row, N);
  MOE_LAUNCH_CHECK();
  return MOE_OK;
}

}  // namespace
}  // namespace moe

using namespace moe;

extern "C" size_t moe_ffn_fwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d, int f,
                                              int64_t rows_alloc) {
  FfnPlan pl;
  return make_plan(dt, act, E, d, f, rows_alloc, pl) ? pl.total_fwd : 0;
}

extern "C" size_t moe_ffn_bwd_workspace_bytes(moe_dtype dt, moe_act act, int E, int d, int f,
                                              int64_t rows_alloc) {
  FfnPlan pl;
  return make_plan(dt, act, E, d, f, rows_alloc, pl) ? pl.total_bwd : 0;
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
  char* abuf = ws + pl.o_abuf;

  GemmParams p = base_params(pl, offsets, ws);
  p.A = static_cast<const char*>(x_disp);
  p.lda = d * es;
  p.B = static_cast<const char*>(w1);
  p.B2 = static_cast<const char*>(w3);
  p.ldb = d * es;
  p.b_gstride = static_cast<int64_t>(f) * d * es;
  p.kbytes = d * es;
  p.N = f;
  p.act = act == MOE_RELU ? ACT_RELU : (act == MOE_GELU_TANH ? ACT_GELU : ACT_SWIGLU);
  p.C = abuf;
  p.ldc = f * es;
  p.H1 = static_cast<char*>(h_save);
  p.H3 = h_save ? static_cast<char*>(h_save) + rows_alloc * f * es : nullptr;
  p.ldh = f * es;
  if (act == MOE_SWIGLU) {
    p.ntiles = cdiv(f, 128);
    MOE_TRY(launch_gemm<M_FWD1_SWIGLU, P_FWD_H>(s, dt, p));
  } else {
    p.ntiles = cdiv(f, BN);
    MOE_TRY(launch_gemm<M_FWD1, P_FWD_H>(s, dt, p));
  }

  GemmParams q = base_params(pl, offsets, ws);
  q.A = abuf;
  q.lda = f * es;
  q.B = static_cast<const char*>(w2);
  q.ldb = f * es;
  q.b_gstride = static_cast<int64_t>(d) * f * es;
  q.kbytes = f * es;
  q.N = d;
  q.ntiles = cdiv(d, BN);
  q.C = static_cast<char*>(y_disp);
  q.ldc = d * es;
  MOE_TRY(launch_gemm<M_STORE, P_FWD_Y>(s, dt, q));
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
  char* w2t = ws + pl.o_w2t;    // [E, f, d]
  char* w13t = ws + pl.o_w13t;  // [E, d, F]
  char* dh = ws + pl.o_dh;      // [rows_alloc, F]
  char* dht = ws + pl.o_dht;    // [F, kpad_cap]
  char* xt = ws + pl.o_xt;      // [d, kpad_cap]
  char* dyt = ws + pl.o_dyt;    // [d, kpad_cap]
  char* at = ws + pl.o_at;      // [f, kpad_cap]
  const int actc = act == MOE_RELU ? ACT_RELU : (act == MOE_GELU_TANH ? ACT_GELU : ACT_SWIGLU);
  const char* h1 = static_cast<const char*>(h_save);
  const char* h3 = sw ? h1 + rows_alloc * f * es : nullptr;

  // weights to K-contiguous form for the data-gradient products
  MOE_TRY(launch_weight_transpose(s, dt, pl, ws, w2, E, d, f, w2t, d, 0,
                                  static_cast<int64_t>(f) * d));
  MOE_TRY(launch_weight_transpose(s, dt, pl, ws, w1, E, f, d, w13t, F, 0,
                                  static_cast<int64_t>(d) * F));
  if (sw)
    MOE_TRY(launch_weight_transpose(s, dt, pl, ws, w3, E, f, d, w13t, F, f,
                                    static_cast<int64_t>(d) * F));

  // dA = dY W2 -> dH (row-major and transposed)
  GemmParams p = base_params(pl, offsets, ws);
  p.A = static_cast<const char*>(dy_disp);
  p.lda = d * es;
  p.B = w2t;
  p.ldb = d * es;
  p.b_gstride = static_cast<int64_t>(f) * d * es;
  p.kbytes = d * es;
  p.N = f;
  p.ntiles = cdiv(f, BN);
  p.act = actc;
  p.C = dh;
  p.ldc = F * es;
  p.H1 = const_cast<char*>(h1);
  p.H3 = const_cast<char*>(h3);
  p.ldh = f * es;
  p.CT = dht;
  p.ldct = static_cast<int64_t>(pl.kpad_cap) * es;
  p.f = f;
  if (sw) MOE_TRY(launch_gemm<M_BWD_DA_SWIGLU, P_BWD_DA>(s, dt, p));
  else MOE_TRY(launch_gemm<M_BWD_DA, P_BWD_DA>(s, dt, p));

  // dx_disp = [dH1 | dH3] [W1 | W3]
  GemmParams q = base_params(pl, offsets, ws);
  q.A = dh;
  q.lda = F * es;
  q.B = w13t;
  q.ldb = F * es;
  q.b_gstride = static_cast<int64_t>(d) * F * es;
  q.kbytes = F * es;
  q.N = d;
  q.ntiles = cdiv(d, BN);
  q.C = static_cast<char*>(dx_disp);
  q.ldc = d * es;
  MOE_TRY(launch_gemm<M_STORE, P_BWD_DX>(s, dt, q));

  // K-contiguous copies of the row operands of the weight gradients
  MOE_TRY(launch_rows_transpose<T_COPY>(s, dt, pl, offsets, ws, x_disp, nullptr, d, 0, xt));
  MOE_TRY(launch_rows_transpose<T_COPY>(s, dt, pl, offsets, ws, dy_disp, nullptr, d, 0, dyt));
  if (sw)
    MOE_TRY(launch_rows_transpose<T_SWIGLU>(s, dt, pl, offsets, ws, h1, h3, f, actc, at));
  else
    MOE_TRY(launch_rows_transpose<T_ACT>(s, dt, pl, offsets, ws, h1, nullptr, f, actc, at));

  // dW2 [d, f] = dY^T A
  GemmParams r = base_params(pl, offsets, ws);
  r.A = dyt;
  r.lda = static_cast<int64_t>(pl.kpad_cap) * es;
  r.M_out = d;
  r.mtiles_out = cdiv(d, BM);
  r.B = at;
  r.ldb = static_cast<int64_t>(pl.kpad_cap) * es;
  r.N = f;
  r.ntiles = cdiv(f, BN);
  r.dwA = dw2;
  r.dwB = dw2;
  r.dw_gstride = static_cast<int64_t>(d) * f;
  r.split_row = d;
  r.partial = reinterpret_cast<float*>(ws + pl.o_part);
  r.slot_elems = static_cast<int64_t>(d) * f;
  MOE_TRY(launch_gemm<M_DW, P_BWD_DW2>(s, dt, r));
  MOE_TRY(launch_split_reduce(s, pl, ws, d, f, dw2, dw2, d));

  // [dW1; dW3] [F, d] = [dH1 dH3]^T X
  GemmParams u = base_params(pl, offsets, ws);
  u.A = dht;
  u.lda = static_cast<int64_t>(pl.kpad_cap) * es;
  u.M_out = F;
  u.mtiles_out = cdiv(F, BM);
  u.B = xt;
  u.ldb = static_cast<int64_t>(pl.kpad_cap) * es;
  u.N = d;
  u.ntiles = cdiv(d, BN);
  u.dwA = dw1;
  u.dwB = sw ? dw3 : dw1;
  u.dw_gstride = static_cast<int64_t>(f) * d;
  u.split_row = f;
  u.partial = reinterpret_cast<float*>(ws + pl.o_part);
  u.slot_elems = static_cast<int64_t>(F) * d;
  MOE_TRY(launch_gemm<M_DW, P_BWD_DW13>(s, dt, u));
  MOE_TRY(launch_split_reduce(s, pl, ws, F, d, dw1, sw ? dw3 : dw1, f));
  return MOE_OK;
}
