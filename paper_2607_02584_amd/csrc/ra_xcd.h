// ra_xcd.h -- XCD-aware placement of attention workgroups (gfx950).
//
// The 256 compute units of an MI355X sit in 8 XCDs, each with its own L2, and
// workgroups are dispatched to the XCDs round-robin in launch order
// (workgroup i -> XCD i % 8).  All query tiles of one head stream the same K/V
// codes, so the tiles are renumbered so that every XCD receives a contiguous
// range of (head, query tile) pairs: the workgroups resident on one XCD then
// share one head's K/V stream in their L2.
#pragma once
#include <hip/hip_runtime.h>

namespace ra {

// Linear launch index -> (head bh, query tile) for a grid of (ntile, nbh).
// A bijection for any grid size: XCD x owns q + (x < r) consecutive tiles,
// q = total / 8, r = total % 8.
__device__ __forceinline__ void xcd_tile(int& bh, int& tile) {
  const int ntile = static_cast<int>(gridDim.x);
  const int total = ntile * static_cast<int>(gridDim.y);
  const int lin = static_cast<int>(blockIdx.x) + ntile * static_cast<int>(blockIdx.y);
  const int q = total >> 3, r = total & 7, x = lin & 7, k = lin >> 3;
  const int L = x * q + (x < r ? x : r) + k;
  bh = L / ntile;
  tile = L - bh * ntile;
}

}  // namespace ra
