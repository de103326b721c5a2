// Host-side argument checks shared by the C entry points.
#pragma once

#include <stdint.h>
#include <stddef.h>

#include "../../include/moe.h"

namespace moe {

constexpr int kMaxE = 64;
constexpr int kMaxRowAlign = 1024;   // largest region alignment of the grouped buffers (rows)
constexpr int kMaxK = 8;

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline bool dtype_ok(moe_dtype dt) { return dt == MOE_F32 || dt == MOE_BF16; }

inline size_t esize(moe_dtype dt) { return dt == MOE_F32 ? 4 : 2; }

// T >= 0, 1 <= E <= 64, 1 <= k <= min(E, 8), T*k < 2^31
inline bool shape_ok(int T, int E, int k) {
  if (T < 0 || E < 1 || E > kMaxE || k < 1 || k > kMaxK || k > E) return false;
  return static_cast<int64_t>(T) * k < (int64_t(1) << 31);
}

// widths: >= 1 and multiples of 8 (16-byte vectors of bf16, 32 bytes of f32)
inline bool width_ok(int d) { return d >= 8 && (d % 8) == 0; }

inline bool rows_ok(int64_t rows_alloc) {
  return rows_alloc >= 0 && rows_alloc < (int64_t(1) << 31);
}

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace moe
