// Debug check of the full pass's layout precondition (include/vtoken.h,
// vtoken_check_layout): every block id of the block tables and the free list lies in the
// pool and appears at most once over both. An admitted request releases all of its blocks
// (Sec. 3.3.3, Sec. 3.3.4), so a block held twice would be released twice (Sec. 3.5, I2).
//
//   layout_clear_kernel    zero the flag word and the one-bit-per-block map
//   layout_mark_kernel     one thread per id: an id outside [0, num_blocks) sets flag bit 0;
//                          an atomicOr that finds the id's bit already set sets flag bit 1
//   layout_finish_kernel   one thread: the status, pool range first, then duplicates
#include "vtoken_internal.h"

namespace vtoken {
namespace {

constexpr int kLayoutThreads = 256;
constexpr int64_t kLayoutMaxGrid = 1 << 16;  // grid-stride beyond

__global__ __launch_bounds__(kLayoutThreads) void layout_clear_kernel(LayoutArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.num_words;
       i += stride) {
    a.words[i] = 0u;
  }
}

__global__ __launch_bounds__(kLayoutThreads) void layout_mark_kernel(LayoutArgs a) {
  const int64_t n = a.num_bt_entries + a.free_len;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  uint32_t* flags = a.words;
  uint32_t* bits = a.words + 1;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int32_t b = i < a.num_bt_entries ? a.block_ids[i] : a.free_list[i - a.num_bt_entries];
    if (static_cast<unsigned>(b) >= static_cast<unsigned>(a.num_blocks)) {
      atomicOr(flags, 1u);
      continue;
    }
    const uint32_t bit = 1u << (b & 31);
    if (atomicOr(bits + (b >> 5), bit) & bit) atomicOr(flags, 2u);
  }
}

__global__ void layout_finish_kernel(LayoutArgs a) {
  if (threadIdx.x != 0) return;
  const uint32_t f = a.words[0];
  a.status[0] = (f & 1u) ? VTOKEN_ERR_BLOCK_RANGE : ((f & 2u) ? VTOKEN_ERR_LAYOUT : VTOKEN_OK);
}

int grid_for(int64_t n) {
  const int64_t g = (n + kLayoutThreads - 1) / kLayoutThreads;
  return static_cast<int>(g < 1 ? 1 : (g > kLayoutMaxGrid ? kLayoutMaxGrid : g));
}

}  // namespace

int64_t layout_words(int32_t num_blocks) { return 1 + ((int64_t)num_blocks + 31) / 32; }

hipError_t launch_check_layout(const LayoutArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(layout_clear_kernel, dim3(grid_for(a.num_words)), dim3(kLayoutThreads), 0,
                     stream, a);
  hipLaunchKernelGGL(layout_mark_kernel, dim3(grid_for(a.num_bt_entries + a.free_len)),
                     dim3(kLayoutThreads), 0, stream, a);
  hipLaunchKernelGGL(layout_finish_kernel, dim3(1), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vtoken
