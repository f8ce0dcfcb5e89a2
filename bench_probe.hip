// Streaming-rate probes of the memory system (gfx950), the measured ceilings the benchmark
// sets the repack and the decode against: plain kernels that read, write or copy large buffers
// in the access patterns of those kernels. Not part of the repack's C ABI (include/vtoken.h):
// a separate library, libvtoken_probe.so, loaded only by `bench.py --mode stream`.
//
// Every kernel gives each 256-thread workgroup one 32 KiB chunk (the size of a (plane, block)
// chunk of the Llama-3-8B copy) and moves it in 16-byte units, eight per thread, all loads of a
// thread issued before any use.
//
//   read         chunk w of the buffer; non-temporal or plain loads
//   write        chunk c(w) = (w % ways) * (chunks / ways) + w / ways: with ways > 1 consecutive
//                workgroups write chunks chunks/ways apart (the repack's block-major order puts
//                consecutive workgroups on one block of different planes); stores through a
//                buffer resource with the repack's cache policy (sc1)
//   copy         chunk c(w) of src to chunk c(w) of dst, non-temporal loads, sc1 stores
//   plane_copy   the repack's work order over contiguous chunks: workgroup w copies a chunk of
//                plane w % planes, consecutive workgroups on different planes
//   head_read    the decode's pattern: 256-byte head pieces of token rows, reached through a slot
//                list, from a K plane and a V plane; workgroup (tile, head) reads the K and V
//                pieces of 64 tokens of one head, grid head-major
//
// The loaded values only feed an XOR that is stored to `sink` when it equals a constant, so
// the loads are kept; a zero-filled buffer never triggers the store (it is in bounds anyway).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnits = 8;                         // 16-byte units per thread
constexpr int64_t kChunk = kThreads * kUnits * 16;  // 32 KiB per workgroup
constexpr uint32_t kBufferDword3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr int kStoreSc1 = 16;                     // the repack's store policy
constexpr uint32_t kSinkKey = 0x9e3779b9u;
constexpr int kHeadPiece = 256;                   // bytes of one head row piece
constexpr int kHeadTokens = 64;                   // tokens per head_read workgroup
constexpr int64_t kMaxGrid = 1 << 24;             // workgroups x 256 threads < 2^32

template <bool kNT>
__device__ __forceinline__ u32x4 load16(const u32x4* p) {
  if constexpr (kNT) {
    return __builtin_nontemporal_load(p);
  } else {
    return *p;
  }
}

__device__ __forceinline__ uint32_t fold(const u32x4* v) {
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < kUnits; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
  return acc;
}

__device__ __forceinline__ int64_t chunk_of(int64_t w, int64_t chunks, int64_t ways) {
  return (w % ways) * (chunks / ways) + w / ways;
}

template <bool kNT>
__global__ __launch_bounds__(kThreads) void probe_read_kernel(const uint8_t* buf,
                                                              uint32_t* sink) {
  const u32x4* base = reinterpret_cast<const u32x4*>(buf + (int64_t)blockIdx.x * kChunk);
  u32x4 v[kUnits];
#pragma unroll
  for (int k = 0; k < kUnits; ++k) v[k] = load16<kNT>(base + k * kThreads + threadIdx.x);
  const uint32_t acc = fold(v);
  if (acc == kSinkKey) sink[0] = acc;
}

__global__ __launch_bounds__(kThreads) void probe_write_kernel(uint8_t* buf, int64_t chunks,
                                                               int64_t ways) {
  uint8_t* base = buf + chunk_of(blockIdx.x, chunks, ways) * kChunk;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(base, 0, static_cast<int>(kChunk), kBufferDword3);
  const u32x4 v = {threadIdx.x, blockIdx.x, 0u, 0u};
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, (k * kThreads + threadIdx.x) * 16, 0,
                                           kStoreSc1);
  }
}

__global__ __launch_bounds__(kThreads) void probe_copy_kernel(const uint8_t* src, uint8_t* dst,
                                                              int64_t chunks, int64_t ways) {
  const int64_t c = chunk_of(blockIdx.x, chunks, ways);
  const u32x4* s = reinterpret_cast<const u32x4*>(src + c * kChunk);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(dst + c * kChunk, 0, static_cast<int>(kChunk),
                                        kBufferDword3);
  u32x4 v[kUnits];
#pragma unroll
  for (int k = 0; k < kUnits; ++k) v[k] = load16<true>(s + k * kThreads + threadIdx.x);
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    __builtin_amdgcn_raw_buffer_store_b128(v[k], rs, (k * kThreads + threadIdx.x) * 16, 0,
                                           kStoreSc1);
  }
}

// The repack's order over contiguous chunks: workgroup w copies chunk src0 + w / planes of plane
// w % planes to chunk dst0 + w / planes of the same plane (consecutive workgroups on one chunk
// index of different planes, as the repack's block-major order puts them), 32 KiB each,
// non-temporal loads and sc1 stores like the repack.
__global__ __launch_bounds__(kThreads) void probe_plane_copy_kernel(uint8_t* base,
                                                                    int64_t plane_bytes,
                                                                    int planes, int64_t src0,
                                                                    int64_t dst0) {
  const int64_t c = blockIdx.x / planes;
  uint8_t* plane = base + (int64_t)(blockIdx.x - c * planes) * plane_bytes;
  const u32x4* s = reinterpret_cast<const u32x4*>(plane + (src0 + c) * kChunk);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      plane + (dst0 + c) * kChunk, 0, static_cast<int>(kChunk), kBufferDword3);
  u32x4 v[kUnits];
#pragma unroll
  for (int k = 0; k < kUnits; ++k) v[k] = load16<true>(s + k * kThreads + threadIdx.x);
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    __builtin_amdgcn_raw_buffer_store_b128(v[k], rs, (k * kThreads + threadIdx.x) * 16, 0,
                                           kStoreSc1);
  }
}

// 16 lanes per 256-byte piece, 16 tokens per pass, 4 passes = 64 tokens; each thread loads
// the K pieces of its 4 tokens, then their V pieces
template <bool kNT>
__global__ __launch_bounds__(kThreads) void probe_head_read_kernel(
    const uint8_t* kv, int64_t plane_bytes, int row_bytes, const int32_t* slots,
    int32_t num_slots, int tiles, uint32_t* sink) {
  const int head = blockIdx.x / tiles;
  const int tile = blockIdx.x - head * tiles;
  const int t_in = threadIdx.x / 16;
  const int col = threadIdx.x % 16;
  const uint8_t* vplane = kv + plane_bytes;
  u32x4 v[kUnits];
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    const int t = tile * kHeadTokens + (k % 4) * 16 + t_in;
    int s = slots[t];
    s = static_cast<unsigned>(s) < static_cast<unsigned>(num_slots) ? s : 0;
    const uint8_t* plane = k < kUnits / 2 ? kv : vplane;
    v[k] = load16<kNT>(reinterpret_cast<const u32x4*>(plane + (int64_t)s * row_bytes +
                                                      (int64_t)head * kHeadPiece) + col);
  }
  const uint32_t acc = fold(v);
  if (acc == kSinkKey) sink[0] = acc;
}

}  // namespace

extern "C" {

// Each call enqueues one kernel on `stream` and returns 0; -2 for a null pointer or a size the
// kernel does not cover (the conditions are stated at each call), -4 for a launch error.

// Read `bytes` of `buf` (a multiple of 32 KiB); nt: non-temporal loads. sink: 4 device bytes.
int vtoken_probe_read(const void* buf, int64_t bytes, int nt, void* sink, hipStream_t stream) {
  if (buf == nullptr || sink == nullptr || bytes <= 0 || bytes % kChunk != 0) return -2;
  const int64_t chunks = bytes / kChunk;
  if (chunks > kMaxGrid) return -2;
  const uint8_t* b = static_cast<const uint8_t*>(buf);
  uint32_t* s = static_cast<uint32_t*>(sink);
  if (nt) {
    hipLaunchKernelGGL(probe_read_kernel<true>, dim3(chunks), dim3(kThreads), 0, stream, b, s);
  } else {
    hipLaunchKernelGGL(probe_read_kernel<false>, dim3(chunks), dim3(kThreads), 0, stream, b, s);
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Write `bytes` of `buf` (a multiple of 32 KiB whose chunk count `ways` divides).
int vtoken_probe_write(void* buf, int64_t bytes, int ways, hipStream_t stream) {
  if (buf == nullptr || bytes <= 0 || bytes % kChunk != 0 || ways <= 0) return -2;
  const int64_t chunks = bytes / kChunk;
  if (chunks > kMaxGrid || chunks % ways != 0) return -2;
  hipLaunchKernelGGL(probe_write_kernel, dim3(chunks), dim3(kThreads), 0, stream,
                     static_cast<uint8_t*>(buf), chunks, (int64_t)ways);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Copy `bytes` from src to dst (non-overlapping; sizes as for vtoken_probe_write).
int vtoken_probe_copy(const void* src, void* dst, int64_t bytes, int ways, hipStream_t stream) {
  if (src == nullptr || dst == nullptr || bytes <= 0 || bytes % kChunk != 0 || ways <= 0) {
    return -2;
  }
  const int64_t chunks = bytes / kChunk;
  if (chunks > kMaxGrid || chunks % ways != 0) return -2;
  hipLaunchKernelGGL(probe_copy_kernel, dim3(chunks), dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(src), static_cast<uint8_t*>(dst), chunks,
                     (int64_t)ways);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// The repack's work order over contiguous chunks: `planes` planes of plane_bytes (a multiple
// of 32 KiB) from `base`; in every plane, chunks [src0, src0 + chunks) are copied to chunks
// [dst0, dst0 + chunks) (both ranges inside the plane, not overlapping).
int vtoken_probe_plane_copy(void* base, int64_t plane_bytes, int planes, int64_t src0,
                            int64_t dst0, int64_t chunks, hipStream_t stream) {
  if (base == nullptr || plane_bytes <= 0 || plane_bytes % kChunk != 0 || planes <= 0 ||
      chunks <= 0 || src0 < 0 || dst0 < 0) {
    return -2;
  }
  const int64_t per_plane = plane_bytes / kChunk;
  if (src0 + chunks > per_plane || dst0 + chunks > per_plane ||
      (src0 < dst0 + chunks && dst0 < src0 + chunks) || chunks * planes > kMaxGrid) {
    return -2;
  }
  hipLaunchKernelGGL(probe_plane_copy_kernel, dim3(static_cast<unsigned>(chunks * planes)),
                     dim3(kThreads), 0, stream, static_cast<uint8_t*>(base), plane_bytes, planes,
                     src0, dst0);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// The decode's pattern: kv holds a K plane and then a V plane of plane_bytes each, token rows
// of row_bytes (a multiple of 256: row_bytes / 256 heads); slots[num_tokens] are row indices
// below plane_bytes / row_bytes (others read row 0); num_tokens a multiple of 64.
int vtoken_probe_head_read(const void* kv, int64_t plane_bytes, int row_bytes,
                           const int32_t* slots, int64_t num_tokens, int nt, void* sink,
                           hipStream_t stream) {
  if (kv == nullptr || slots == nullptr || sink == nullptr || row_bytes <= 0 ||
      row_bytes % kHeadPiece != 0 || num_tokens <= 0 || num_tokens % kHeadTokens != 0 ||
      plane_bytes < (int64_t)row_bytes) {
    return -2;
  }
  const int64_t rows = plane_bytes / row_bytes;
  const int heads = row_bytes / kHeadPiece;
  const int64_t tiles = num_tokens / kHeadTokens;
  if (rows > 0x7fffffff || tiles * heads > kMaxGrid) return -2;
  const uint8_t* b = static_cast<const uint8_t*>(kv);
  uint32_t* s = static_cast<uint32_t*>(sink);
  const dim3 grid(static_cast<unsigned>(tiles * heads));
  if (nt) {
    hipLaunchKernelGGL(probe_head_read_kernel<true>, grid, dim3(kThreads), 0, stream, b,
                       plane_bytes, row_bytes, slots, static_cast<int32_t>(rows),
                       static_cast<int>(tiles), s);
  } else {
    hipLaunchKernelGGL(probe_head_read_kernel<false>, grid, dim3(kThreads), 0, stream, b,
                       plane_bytes, row_bytes, slots, static_cast<int32_t>(rows),
                       static_cast<int>(tiles), s);
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
