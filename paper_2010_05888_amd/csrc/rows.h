// Where the streaming kernels find the n vectors they read: the rows of one
// row-major n x d matrix, or a table of row pointers -- one segment of n
// vectors stored apart (the same layer's gradient from each of n workers, or
// n whole vectors in separate buffers).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace garfield {

struct MatrixRows {
  const float* x;
  int64_t d;
  __device__ __forceinline__ const float* row(int64_t i) const { return x + i * d; }
};

struct TableRows {
  const float* const* p;  // p[i] = vector i's segment
  __device__ __forceinline__ const float* row(int64_t i) const { return p[i]; }
};

// A batch of segments for one launch, passed by value in the kernel
// arguments: each segment's length, the coordinates one of its workgroups
// covers, its first workgroup and, for the aggregation kernels, its output.
// Workgroup b works on the segment s with first[s] <= b < first[s + 1].
constexpr int kSegMax = 96;
struct SegTable {
  int count;
  int32_t first[kSegMax + 1];  // first[count] = workgroups of the launch
  int32_t span[kSegMax];
  int64_t dims[kSegMax];
  float* outs[kSegMax];
};

// The segment of workgroup b: the largest s with first[s] <= b (empty segments
// share their start with the next one and are skipped).
__device__ __forceinline__ int seg_of(const SegTable& t, int b) {
  int lo = 0, hi = t.count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (t.first[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

}  // namespace garfield
