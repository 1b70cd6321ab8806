// Workgroup-to-tile mapping that keeps neighbouring tiles on one XCD.
//
// The dispatcher hands workgroup i (linear id over the grid) to XCD i mod 8,
// and each XCD has its own L2.  Tiles that share an operand (the column units
// of one row block read the same rows of the projection) should run on the
// same XCD at about the same time, so that the second and later reads hit
// that XCD's L2.  xcd_tile maps the linear workgroup id to a logical tile id
// such that XCD x runs one contiguous range of logical ids, in order: with
// total = 8 q + rem, XCDs below rem take q + 1 ids, the others q.  It is a
// bijection on [0, total).
#pragma once

#include <stdint.h>

namespace gift {

constexpr int kXcdCount = 8;

__device__ __forceinline__ int64_t xcd_tile(int64_t lin, int64_t total) {
  const int64_t q = total / kXcdCount, rem = total % kXcdCount;
  const int64_t x = lin % kXcdCount, k = lin / kXcdCount;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + k;
}

}  // namespace gift
