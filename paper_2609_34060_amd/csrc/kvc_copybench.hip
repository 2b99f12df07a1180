// Copy ceilings of the apply's memory traffic on this GPU (measurement only; not part of the correction path).
//
// The apply reads each source row once and writes each destination row once through shuffled block tables, so its
// rate is bounded by what a plain copy with the same access pattern reaches.  These kernels move bytes only, with the
// same 16-byte accesses as the apply:
//   contiguous    one buffer to another, grid-stride or one contiguous chunk per workgroup (optionally ordered so
//                 that the workgroups of one XCD stream one contiguous range: the hardware hands workgroup i to
//                 XCD i mod 8)
//   read / write  read-only and write-only streams of one buffer
//   paged_blocks  whole blocks through a source and a destination table, in a caller-given work order (entry i of
//                 `order` is the logical block workgroup i takes)
//   paged_heads   the apply's own pattern: one KV head's rows of consecutive logical blocks per workgroup
// Launch sizes are checked on the host: every kernel reads and writes only inside the element counts it is given.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;  // 16-byte loads in flight per thread

__global__ __launch_bounds__(kThreads) void copy_gridstride(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                            int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = src[i + u * stride];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) dst[i + u * stride] = v[u];
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

// Workgroup b copies chunk c(b) of n / gridDim.x elements; with xcd_order the eight XCDs each take one contiguous
// eighth of the chunks (workgroup b runs on XCD b mod 8).
__global__ __launch_bounds__(kThreads) void copy_chunked(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                         int64_t n, int xcd_order) {
  const int64_t nwg = gridDim.x, b = blockIdx.x;
  const int64_t c = xcd_order ? (b % 8) * (nwg / 8) + b / 8 : b;
  const int64_t per = n / nwg, begin = c * per, end = c == nwg - 1 ? n : begin + per;
  int64_t i = begin + threadIdx.x;
  for (; i + (kUnroll - 1) * kThreads < end; i += kUnroll * kThreads) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = src[i + u * kThreads];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) dst[i + u * kThreads] = v[u];
  }
  for (; i < end; i += kThreads) dst[i] = src[i];
}

// Read-only stream: every element is read once; the xor of all of them is written only if it equals `never` (the
// caller passes a value that does not occur), so the loads are kept and nothing is stored.
__global__ __launch_bounds__(kThreads) void read_stream(const u32x4* __restrict__ src, int64_t n, uint32_t never,
                                                        uint32_t* __restrict__ sink, int xcd_order) {
  const int64_t nwg = gridDim.x, b = blockIdx.x;
  const int64_t c = xcd_order ? (b % 8) * (nwg / 8) + b / 8 : b;
  const int64_t per = n / nwg, begin = c * per, end = c == nwg - 1 ? n : begin + per;
  u32x4 acc = {0u, 0u, 0u, 0u};
  int64_t i = begin + threadIdx.x;
  for (; i + (kUnroll - 1) * kThreads < end; i += kUnroll * kThreads) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = src[i + u * kThreads];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
  }
  for (; i < end; i += kThreads) acc ^= src[i];
  const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (x == never) sink[0] = x;
}

__global__ __launch_bounds__(kThreads) void write_stream(u32x4* __restrict__ dst, int64_t n, uint32_t value,
                                                         int xcd_order) {
  const int64_t nwg = gridDim.x, b = blockIdx.x;
  const int64_t c = xcd_order ? (b % 8) * (nwg / 8) + b / 8 : b;
  const int64_t per = n / nwg, begin = c * per, end = c == nwg - 1 ? n : begin + per;
  const u32x4 v = {value, value, value, value};
  for (int64_t i = begin + threadIdx.x; i < end; i += kThreads) dst[i] = v;
}

// Whole blocks: workgroup i copies `blocks_per_wg` logical blocks order[i * blocks_per_wg + j] from physical block
// src_table[l] to dst_table[l]; a block is `block_elems` 16-byte elements.
__global__ __launch_bounds__(kThreads) void paged_blocks(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                         const int32_t* __restrict__ src_table,
                                                         const int32_t* __restrict__ dst_table,
                                                         const int32_t* __restrict__ order, int num_blocks,
                                                         int blocks_per_wg, int block_elems) {
  for (int j = 0; j < blocks_per_wg; ++j) {
    const int64_t slot = (int64_t)blockIdx.x * blocks_per_wg + j;
    if (slot >= num_blocks) return;
    const int l = order[slot];
    const u32x4* s = src + (int64_t)src_table[l] * block_elems;
    u32x4* d = dst + (int64_t)dst_table[l] * block_elems;
    int e = threadIdx.x;
    for (; e + (kUnroll - 1) * kThreads < block_elems; e += kUnroll * kThreads) {
      u32x4 v[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) v[u] = s[e + u * kThreads];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) d[e + u * kThreads] = v[u];
    }
    for (; e < block_elems; e += kThreads) d[e] = s[e];
  }
}

// The apply's pattern: workgroup (chunk, head) copies head `head`'s rows of the `tokens_per_wg` tokens starting at
// chunk * tokens_per_wg; a token row is row_elems 16-byte elements (16 per 256-byte row), tokens sit at
// token_elems strides inside a block of block_tokens tokens.
__global__ __launch_bounds__(kThreads) void paged_heads(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                        const int32_t* __restrict__ src_table,
                                                        const int32_t* __restrict__ dst_table, int num_tokens,
                                                        int tokens_per_wg, int block_tokens, int block_elems,
                                                        int token_elems, int row_elems) {
  const int head = blockIdx.y;
  const int t0 = blockIdx.x * tokens_per_wg, t1 = min(num_tokens, t0 + tokens_per_wg);
  const int rows_per_pass = kThreads / row_elems;
  const int sub = threadIdx.x / row_elems, e = threadIdx.x % row_elems;
  for (int t = t0 + sub; t < t1; t += kUnroll * rows_per_pass) {
    u32x4 v[kUnroll];
    int64_t so[kUnroll], dof[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int tt = t + u * rows_per_pass;
      so[u] = dof[u] = -1;
      if (tt < t1) {
        const int lb = tt / block_tokens, slot = tt - lb * block_tokens;
        const int64_t in_block = (int64_t)slot * token_elems + (int64_t)head * row_elems + e;
        so[u] = (int64_t)src_table[lb] * block_elems + in_block;
        dof[u] = (int64_t)dst_table[lb] * block_elems + in_block;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (so[u] >= 0) v[u] = src[so[u]];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (dof[u] >= 0) dst[dof[u]] = v[u];
  }
}

}  // namespace

extern "C" {

// All sizes in 16-byte elements; pointers are device memory of at least the stated extent.  Returns hipError_t.
int kvcb_copy(const void* src, void* dst, int64_t n, int workgroups, int mode, hipStream_t stream) {
  if (n <= 0 || workgroups < 8 || workgroups % 8) return (int)hipErrorInvalidValue;
  const u32x4* s = static_cast<const u32x4*>(src);
  u32x4* d = static_cast<u32x4*>(dst);
  if (mode == 0)
    hipLaunchKernelGGL(copy_gridstride, dim3(workgroups), dim3(kThreads), 0, stream, s, d, n);
  else
    hipLaunchKernelGGL(copy_chunked, dim3(workgroups), dim3(kThreads), 0, stream, s, d, n, mode == 2 ? 1 : 0);
  return (int)hipGetLastError();
}

int kvcb_read(const void* src, int64_t n, int workgroups, int xcd_order, uint32_t never, void* sink,
              hipStream_t stream) {
  if (n <= 0 || workgroups < 8 || workgroups % 8) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(read_stream, dim3(workgroups), dim3(kThreads), 0, stream, static_cast<const u32x4*>(src), n,
                     never, static_cast<uint32_t*>(sink), xcd_order);
  return (int)hipGetLastError();
}

int kvcb_write(void* dst, int64_t n, int workgroups, int xcd_order, uint32_t value, hipStream_t stream) {
  if (n <= 0 || workgroups < 8 || workgroups % 8) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(write_stream, dim3(workgroups), dim3(kThreads), 0, stream, static_cast<u32x4*>(dst), n, value,
                     xcd_order);
  return (int)hipGetLastError();
}

// src / dst: pools of at least max(table entry) + 1 blocks; tables and order: device int32 [num_blocks], order a
// permutation of 0 .. num_blocks - 1.
int kvcb_paged_blocks(const void* src, void* dst, const int32_t* src_table, const int32_t* dst_table,
                      const int32_t* order, int num_blocks, int blocks_per_wg, int block_elems, hipStream_t stream) {
  if (num_blocks <= 0 || blocks_per_wg <= 0 || block_elems <= 0) return (int)hipErrorInvalidValue;
  const int wgs = (num_blocks + blocks_per_wg - 1) / blocks_per_wg;
  hipLaunchKernelGGL(paged_blocks, dim3(wgs), dim3(kThreads), 0, stream, static_cast<const u32x4*>(src),
                     static_cast<u32x4*>(dst), src_table, dst_table, order, num_blocks, blocks_per_wg, block_elems);
  return (int)hipGetLastError();
}

// tables: device int32 [ceil(num_tokens / block_tokens)]; heads * row_elems <= token_elems,
// block_tokens * token_elems <= block_elems, row_elems divides 256.
int kvcb_paged_heads(const void* src, void* dst, const int32_t* src_table, const int32_t* dst_table, int num_tokens,
                     int heads, int tokens_per_wg, int block_tokens, int block_elems, int token_elems, int row_elems,
                     hipStream_t stream) {
  if (num_tokens <= 0 || heads <= 0 || tokens_per_wg <= 0 || row_elems <= 0 || kThreads % row_elems ||
      heads * row_elems > token_elems || block_tokens * token_elems > block_elems)
    return (int)hipErrorInvalidValue;
  dim3 grid((num_tokens + tokens_per_wg - 1) / tokens_per_wg, heads);
  hipLaunchKernelGGL(paged_heads, grid, dim3(kThreads), 0, stream, static_cast<const u32x4*>(src),
                     static_cast<u32x4*>(dst), src_table, dst_table, num_tokens, tokens_per_wg, block_tokens,
                     block_elems, token_elems, row_elems);
  return (int)hipGetLastError();
}

}  // extern "C"
