// Host-side argument checks shared by the C-ABI entry points.
#pragma once

#include <cstdint>

namespace dsa3d {
namespace api {

struct Span {
  uintptr_t lo, hi;  // [lo, hi)
};

inline bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

inline bool aligned(const void* p, uintptr_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

inline Span span_of(const void* p, uint64_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return Span{lo, lo + bytes};
}

}  // namespace api
}  // namespace dsa3d
