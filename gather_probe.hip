// Gather-bandwidth microbenchmark (measurement only; not part of the operator library; built
// beside bench.py, which reports its figures).
//
// The 3D-DSA kernels read their K/V corner rows (and the backward its q/dout rows) as 16-byte
// loads per lane in which each group of L lanes covers one contiguous row at an unrelated
// address.  This probe measures how many bytes per clock one compute unit can gather in that
// pattern when every row already sits in the unit's vector L1 cache (a 16 KB working set per
// workgroup), and, for comparison, from LDS (ds_read_b128 into a 64 KB LDS array).  The L1
// figure is the ceiling of the operator's gather path: a kernel whose rows also miss L1 can
// only be slower.  A third mode reads rows at random from a 2 MB region shared by all
// workgroups: it misses L1 and hits L2, the rate of rows that the vector L1 does not hold.
// A fourth reads them from a 512 MB region, twice the memory-side cache: almost every row
// misses L2, the rate at which rows come from past the L2s.  Two more modes gather the
// L1-resident and the L2-resident rows with gfx950's direct-to-LDS loads
// (global_load_lds_dwordx4: each lane's 16 bytes land in LDS, not in registers) and then read
// them from LDS, eight loads per wave in flight, to see whether that path takes rows faster.
//
// Every index is masked into its buffer: lds_gather touches slots [0, 4096) of its 64 KB
// array, l1_gather slots [0, 1024) of its block's 16 KB region of the source buffer, whose
// 256 regions the host allocates (4 MB), l2_gather slots [0, 131072) of that buffer, and
// mem_gather slots [0, 2^25) of the 512 MB buffer the host allocates for it; to_lds_gather
// reads the slots of l1_gather or l2_gather and writes, per wave, 8 x 64 slots of its 32 KB LDS
// array.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
constexpr int kLdsSlots = 65536 / 16;  // 16-byte slots of the LDS array
constexpr int kL1Slots = 16384 / 16;   // 16-byte slots of one block's L1-resident region
constexpr int kRegions = 256;
constexpr int kL2Slots = (2 << 20) / 16;  // 16-byte slots of the L2-resident region
constexpr int kMemSlots = (512 << 20) / 16;  // 16-byte slots of the region past the L2s

template <int GS>
__global__ __launch_bounds__(kThreads) void lds_gather(uint4* out, int iters, uint32_t seed) {
  __shared__ uint4 buf[kLdsSlots];
  for (int i = threadIdx.x; i < kLdsSlots; i += kThreads) buf[i] = make_uint4(i, i + 1, i + 2, i + 3);
  __syncthreads();
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    h = h * 1664525u + 1013904223u;
    const uint32_t idx = ((h >> 8) & (kLdsSlots / GS - 1)) * GS + part;
    const uint4 v = buf[idx];
    acc.x ^= v.x;
    acc.y += v.y;
    acc.z ^= v.z;
    acc.w += v.w;
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

template <int GS>
__global__ __launch_bounds__(kThreads) void l1_gather(const uint4* __restrict__ src, uint4* out,
                                                      int iters, uint32_t seed) {
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  const uint4* base = src + (blockIdx.x % kRegions) * kL1Slots;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    h = h * 1664525u + 1013904223u;
    const uint32_t idx = ((h >> 8) & (kL1Slots / GS - 1)) * GS + part;
    const uint4 v = base[idx];
    acc.x ^= v.x;
    acc.y += v.y;
    acc.z ^= v.z;
    acc.w += v.w;
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

template <int GS>
__global__ __launch_bounds__(kThreads) void l2_gather(const uint4* __restrict__ src, uint4* out,
                                                      int iters, uint32_t seed) {
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    h = h * 1664525u + 1013904223u;
    const uint32_t idx = ((h >> 4) & (kL2Slots / GS - 1)) * GS + part;
    const uint4 v = src[idx];
    acc.x ^= v.x;
    acc.y += v.y;
    acc.z ^= v.z;
    acc.w += v.w;
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

template <int GS>
__global__ __launch_bounds__(kThreads) void mem_gather(const uint4* __restrict__ src, uint4* out,
                                                       int iters, uint32_t seed) {
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    h = h * 1664525u + 1013904223u;
    const uint32_t idx = ((h >> 4) & (kMemSlots / GS - 1)) * GS + part;
    const uint4 v = src[idx];
    acc.x ^= v.x;
    acc.y += v.y;
    acc.z ^= v.z;
    acc.w += v.w;
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

// The gathers of l1_gather (L2 = false) and l2_gather (L2 = true) through direct-to-LDS
// loads: per outer step each wave issues 8 of them into its 8 x 1 KB of LDS (the lanes' 16-byte
// pieces in lane order), waits for them and reads its lane's 8 pieces back.  iters is a
// multiple of 8.
template <int GS, bool L2>
__global__ __launch_bounds__(kThreads) void to_lds_gather(const uint4* __restrict__ src, uint4* out,
                                                          int iters, uint32_t seed) {
  constexpr int kInFlight = 8;
  __shared__ uint4 buf[kThreads / 64][kInFlight][64];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  const uint4* base = L2 ? src : src + (blockIdx.x % kRegions) * kL1Slots;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
  for (int it = 0; it < iters; it += kInFlight) {
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      h = h * 1664525u + 1013904223u;
      const uint32_t idx = L2 ? ((h >> 4) & (kL2Slots / GS - 1)) * GS + part
                              : ((h >> 8) & (kL1Slots / GS - 1)) * GS + part;
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(base + idx),
                                       (__attribute__((address_space(3))) void*)&buf[wave][u][0],
                                       16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the wave's LDS pieces have landed
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const uint4 v = buf[wave][u][lane];
      acc.x ^= v.x;
      acc.y += v.y;
      acc.z ^= v.z;
      acc.w += v.w;
    }
    __builtin_amdgcn_s_waitcnt(0);  // read before the next step's loads overwrite them
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

// Rows of GS * 16 bytes drawn at random from `nrows` rows laid out `stride16` 16-byte slots
// apart (the rows of one head of a [token][heads][head_dim] tensor are heads * row bytes
// apart): the working set is nrows * GS * 16 bytes, the span nrows * stride16 * 16.
template <int GS>
__global__ __launch_bounds__(kThreads) void set_gather(const uint4* __restrict__ src, uint4* out,
                                                       int iters, uint32_t seed, uint32_t nrows,
                                                       uint32_t stride16) {
  uint32_t h = (threadIdx.x / GS) * 2654435761u + seed + blockIdx.x * 97u;
  const int part = threadIdx.x % GS;
  uint4 acc = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll 8
  for (int it = 0; it < iters; ++it) {
    h = h * 1664525u + 1013904223u;
    const uint32_t row = (uint32_t)(((uint64_t)h * nrows) >> 32);  // < nrows
    const uint4 v = src[(uint64_t)row * stride16 + part];
    acc.x ^= v.x;
    acc.y += v.y;
    acc.z ^= v.z;
    acc.w += v.w;
  }
  out[blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

// Gathers rows of `row_bytes` (128 or 256) at random from a working set of `set_bytes`
// (whole rows) whose rows are `stride_bytes` apart (a multiple of 16, at least row_bytes;
// the span set_bytes / row_bytes * stride_bytes at most 4 GB), over `blocks` workgroups of
// `iters` loads per lane, twice; stores the second run's time in *ms and the bytes gathered
// per run in *bytes.  Shows how the rate falls once the set outgrows an XCD's L2.  Returns 0,
// a nonzero hipError_t, or -1 for arguments outside those values.  Allocates and frees its
// own buffers and synchronises the device.
int dsa3d_probe_working_set(int row_bytes, long long stride_bytes, long long set_bytes,
                            int blocks, int iters, float* ms, double* bytes) {
  if (ms == nullptr || bytes == nullptr || blocks < 1 || iters < 1) return -1;
  if ((row_bytes != 128 && row_bytes != 256) || stride_bytes < row_bytes ||
      stride_bytes % 16 != 0 || set_bytes < row_bytes)
    return -1;
  const long long nrows = set_bytes / row_bytes;
  const long long span = nrows * stride_bytes;
  if (nrows >= (1ll << 32) || span > (4ll << 30)) return -1;
  const void* fn = row_bytes == 256 ? (const void*)&set_gather<16> : (const void*)&set_gather<8>;
  uint4 *out = nullptr, *src = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipMalloc(&out, (size_t)blocks * kThreads * sizeof(uint4));
  if (e == hipSuccess) e = hipMalloc(&src, (size_t)span);
  if (e == hipSuccess) e = hipMemset(src, 1, (size_t)span);
  if (e == hipSuccess) e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  uint32_t nr = (uint32_t)nrows, s16 = (uint32_t)(stride_bytes / 16);
  for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {
    uint32_t seed = 7u + rep;
    void* args[] = {(void*)&src, (void*)&out, (void*)&iters, (void*)&seed, (void*)&nr, (void*)&s16};
    e = hipEventRecord(a, 0);
    if (e == hipSuccess) e = hipLaunchKernel(fn, dim3(blocks), dim3(kThreads), args, 0, 0);
    if (e == hipSuccess) e = hipEventRecord(b, 0);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    if (e == hipSuccess) e = hipEventElapsedTime(ms, a, b);
  }
  *bytes = (double)blocks * kThreads * (double)iters * 16.0;
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (src) (void)hipFree(src);
  if (out) (void)hipFree(out);
  return (int)e;
}


// Runs the gather of `source` (0: L1-resident global loads, 1: LDS, 2: global loads that miss
// L1 and hit L2, 3: global loads that miss L2, 4 and 5: the rows of 0 and 2 through
// direct-to-LDS loads, read back from LDS) with row pieces of
// `row_bytes` (32, 64, 128 or 256: GS = row_bytes / 16 lanes per row) over `blocks`
// workgroups of `iters` loads per lane (a multiple of 8 for sources 4 and 5), twice; stores
// the second run's time in *ms and the bytes gathered per run in *bytes.  Returns 0, or a
// nonzero hipError_t / -1 for arguments outside those values.  Allocates and frees its own
// buffers and synchronises the device.
int dsa3d_probe_gather(int source, int row_bytes, int blocks, int iters, float* ms,
                       double* bytes) {
  if (ms == nullptr || bytes == nullptr || blocks < 1 || iters < 1 || source < 0 || source > 5 ||
      (source >= 4 && iters % 8 != 0))
    return -1;
  const void* fns[4][6] = {
      {(const void*)&l1_gather<2>, (const void*)&lds_gather<2>, (const void*)&l2_gather<2>,
       (const void*)&mem_gather<2>, (const void*)&to_lds_gather<2, false>,
       (const void*)&to_lds_gather<2, true>},
      {(const void*)&l1_gather<4>, (const void*)&lds_gather<4>, (const void*)&l2_gather<4>,
       (const void*)&mem_gather<4>, (const void*)&to_lds_gather<4, false>,
       (const void*)&to_lds_gather<4, true>},
      {(const void*)&l1_gather<8>, (const void*)&lds_gather<8>, (const void*)&l2_gather<8>,
       (const void*)&mem_gather<8>, (const void*)&to_lds_gather<8, false>,
       (const void*)&to_lds_gather<8, true>},
      {(const void*)&l1_gather<16>, (const void*)&lds_gather<16>, (const void*)&l2_gather<16>,
       (const void*)&mem_gather<16>, (const void*)&to_lds_gather<16, false>,
       (const void*)&to_lds_gather<16, true>}};
  int ri;
  switch (row_bytes) {
    case 32: ri = 0; break;
    case 64: ri = 1; break;
    case 128: ri = 2; break;
    case 256: ri = 3; break;
    default: return -1;
  }
  const void* fn = fns[ri][source];
  uint4 *out = nullptr, *src = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  const size_t src_bytes = (source == 3 ? (size_t)kMemSlots : (size_t)kRegions * kL1Slots) * 16;
  hipError_t e = hipMalloc(&out, (size_t)blocks * kThreads * sizeof(uint4));
  if (e == hipSuccess) e = hipMalloc(&src, src_bytes);
  if (e == hipSuccess) e = hipMemset(src, 1, src_bytes);
  if (e == hipSuccess) e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {
    uint32_t seed = 1u + rep;
    void* args_l1[] = {(void*)&src, (void*)&out, (void*)&iters, (void*)&seed};
    void* args_lds[] = {(void*)&out, (void*)&iters, (void*)&seed};
    e = hipEventRecord(a, 0);
    if (e == hipSuccess)
      e = hipLaunchKernel(fn, dim3(blocks), dim3(kThreads), source == 1 ? args_lds : args_l1, 0, 0);
    if (e == hipSuccess) e = hipEventRecord(b, 0);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    if (e == hipSuccess) e = hipEventElapsedTime(ms, a, b);
  }
  *bytes = (double)blocks * kThreads * (double)iters * 16.0;
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (src) (void)hipFree(src);
  if (out) (void)hipFree(out);
  return (int)e;
}

}  // extern "C"
