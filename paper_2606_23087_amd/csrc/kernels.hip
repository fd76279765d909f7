// HIP kernels of libflowpool for gfx950 (CDNA4).
//
// k_pack  : the consumer's translate-gather-pack of one microbatch
//           (paper Sec. 3.1 / Sec. 3.2): prefix sum of sample lengths ->
//           cu_seqlens; per row, the sample and its text/image segment; for
//           image rows the GVA page walk through the page table; then 16-byte
//           vector copies of every row from its page or embedding-table row
//           into the packed output, plus position ids.
// k_write : the producer's write of one sample's image rows into its pages,
//           through the same page table (Sec. 3.2, producer side), and
//           publication of the sample descriptor.
// k_cost  : per-sample cost K*l + l^2 for the planner (Sec. 3.4).
//
// Nothing here is a dense contraction, so there is no MFMA: the pack is a
// bandwidth-bound gather whose cost is HBM bytes.

#include "fp_internal.h"

namespace fp {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Global-address-space views: loads through them compile to global_load
// (vector memory counter only) instead of flat loads, which also count
// against the LDS counter and force the compiler to wait for each one.
typedef __attribute__((address_space(1))) const u32x4 g_u32x4_c;
typedef __attribute__((address_space(1))) u32x4 g_u32x4;

__device__ __forceinline__ u32x4 load16(const uint8_t* p) {
  return __builtin_nontemporal_load((g_u32x4_c*)p);
}

__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, (g_u32x4*)p);
}

template <typename T>
__device__ __forceinline__ T ld_global(const T* p) {
  return *(const __attribute__((address_space(1))) T*)p;
}

__device__ __forceinline__ PackSample ld_sample(const PackSample* p) {
  const g_u32x4_c* q = (const g_u32x4_c*)p;
  const u32x4 lo = q[0], hi = q[1];
  PackSample s;
  __builtin_memcpy(&s, &lo, 16);
  __builtin_memcpy(reinterpret_cast<uint8_t*>(&s) + 16, &hi, 16);
  return s;
}

__device__ __forceinline__ int2 ld_pair(const int2* p) {
  const uint64_t v = ld_global(reinterpret_cast<const uint64_t*>(p));
  int2 r;
  r.x = (int)(uint32_t)v;
  r.y = (int)(uint32_t)(v >> 32);
  return r;
}

// Block-wide exclusive prefix sum of len[0..n) into cu[0..n] (cu[0] = 0).
__device__ __forceinline__ void block_scan_lengths(const PackSample* smp, int n, int32_t* cu,
                                                   int32_t* wsum) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) cu[0] = 0;
  int carry = 0;
  for (int base = 0; base < n; base += kBlock) {
    const int i = base + tid;
    int v = (i < n) ? smp[i].len : 0;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(v, d, 64);
      if (lane >= d) v += t;
    }
    if (lane == 63) wsum[wave] = v;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kBlock / 64; ++w) {
      before += (w < wave) ? wsum[w] : 0;
      all += wsum[w];
    }
    if (i < n) cu[i + 1] = carry + before + v;
    carry += all;
    __syncthreads();
  }
}

// Index of the sample holding packed row `row`: last k with cu[k] <= row.
__device__ __forceinline__ int sample_of(const int32_t* cu, int n, int row) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Source address of row r of sample sp (null if the tier mask skips it).
__device__ __forceinline__ const uint8_t* resolve_row(const PackArgs& a, const PackSample& sp,
                                                      const int2* img, int r) {
  // Image j of the sample starts after img.x of its text rows and all rows
  // of the images before it; text rows fill the gaps.
  int vis_before = 0, vis_idx = -1;
  for (int j = 0; j < sp.n_img; ++j) {
    const int2 pr = img[sp.img_base + j];
    const int start = pr.x + vis_before;
    if (r < start) break;
    if (r < start + pr.y) { vis_idx = vis_before + (r - start); break; }
    vis_before += pr.y;
  }
  if (vis_idx < 0) {
    if (!(a.tier_mask & 1)) return nullptr;
    const int32_t id = ld_global(reinterpret_cast<const int32_t*>(a.meta + sp.text_off) + (r - vis_before));
    return a.table + (size_t)id * a.row_bytes;
  }
  // Page walk: visual row -> page GVA -> page-table entry -> physical row.
  const int lp = vis_idx / a.page_tokens;
  const int off = vis_idx - lp * a.page_tokens;
  const uint64_t gva = ld_global(reinterpret_cast<const uint64_t*>(a.meta + sp.page_off) + lp);
  const uint64_t pte = ld_global(a.pte + (gva - a.gva_start) / a.page_bytes);
  if (!(a.tier_mask & ((pte & PTE_HOST) ? 2 : 1))) return nullptr;
  return reinterpret_cast<const uint8_t*>(pte & PTE_ADDR_MASK) + (size_t)off * a.row_bytes;
}

// One workgroup packs one chunk of kChunkVecs 16-byte vectors of the output
// (rows are contiguous in the output, so a chunk is a contiguous byte range
// that may start and end inside rows): it stages the microbatch's sample
// headers in LDS, computes the prefix sum of their lengths, resolves the
// source of every row the chunk touches, then moves kVecsPerThread vectors
// per thread with all loads in flight before the stores.
__global__ __launch_bounds__(kBlock) void k_pack(PackArgs a) {
  extern __shared__ __align__(16) uint8_t s_dyn[];
  __shared__ int32_t s_wsum[kBlock / 64];
  __shared__ int32_t s_skip;                        // some row of the chunk is not copied
  PackSample* s_smp = reinterpret_cast<PackSample*>(s_dyn);
  int2* s_img = reinterpret_cast<int2*>(s_smp + a.n);
  uint64_t* s_src = reinterpret_cast<uint64_t*>(s_img + a.n_imgs);
  int32_t* s_cu = reinterpret_cast<int32_t*>(s_src + a.max_chunk_rows);
  const int tid = threadIdx.x;

  if (tid == 0) s_skip = 0;
  const PackSample* gs = a.samples_dev ? a.samples_dev : a.samples;
  const int2* gi = a.imgs_dev ? a.imgs_dev : a.imgs;
  for (int i = tid; i < a.n; i += kBlock) s_smp[i] = ld_sample(gs + i);
  for (int i = tid; i < a.n_imgs; i += kBlock) s_img[i] = ld_pair(gi + i);
  __syncthreads();
  block_scan_lengths(s_smp, a.n, s_cu, s_wsum);

  const bool write_meta = (a.tier_mask & 1) != 0;
  if (blockIdx.x == 0 && a.cu && write_meta) {
    for (int i = tid; i <= a.n; i += kBlock) a.cu[i] = s_cu[i];
  }

  const int vpr = a.row_bytes >> 4;
  const int total = a.n_tokens * vpr;                 // the host keeps this below 2^31
  const int v0 = blockIdx.x * kChunkVecs;
  const int v1 = min(v0 + kChunkVecs, total);
  const int r0 = v0 / vpr;
  const int rows = v1 > v0 ? (v1 - 1) / vpr - r0 + 1 : 0;
  for (int t = tid; t < rows; t += kBlock) {
    const int row = r0 + t;
    const int k = sample_of(s_cu, a.n, row);
    const int r = row - s_cu[k];
    const uint8_t* src = resolve_row(a, s_smp[k], s_img, r);
    s_src[t] = reinterpret_cast<uint64_t>(src);
    if (!src) s_skip = 1;
    if (a.pos && write_meta && row * vpr >= v0) a.pos[row] = r;
  }
  __syncthreads();

  // Vector e of the chunk belongs to row e / vpr (multiply-shift division).
  // A vector is live if it lies in the chunk and its row is copied; only
  // live vectors get an address, dead ones are never loaded or stored.
  uint64_t from[kVecsPerThread];
  bool live[kVecsPerThread];
#pragma unroll
  for (int u = 0; u < kVecsPerThread; ++u) {
    const int e = v0 + u * kBlock + tid;
    from[u] = 0;
    live[u] = false;
    if (e < v1) {
      const int row = (int)(((uint64_t)(uint32_t)e * a.div_mul) >> a.div_shift);
      const uint64_t base = s_src[row - r0];
      live[u] = base != 0;
      from[u] = live[u] ? base + (uint64_t)(e - row * vpr) * 16 : 0;
    }
  }
  u32x4 v[kVecsPerThread];
  if (v1 - v0 == kChunkVecs && !s_skip) {
    // Whole chunk, every row copied: no predication, so the compiler can keep
    // all loads in flight and wait for them one at a time before each store.
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u) v[u] = load16(reinterpret_cast<const uint8_t*>(from[u]));
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      store16(a.out + (size_t)(v0 + u * kBlock + tid) * 16, v[u]);
  } else {
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      if (live[u]) v[u] = load16(reinterpret_cast<const uint8_t*>(from[u]));
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      if (live[u]) store16(a.out + (size_t)(v0 + u * kBlock + tid) * 16, v[u]);
  }
}

template <int U>
__global__ __launch_bounds__(kBlock) void k_write(WriteArgs a) {
  __shared__ uint8_t* s_dst[kMaxTileRows];
  const int tid = threadIdx.x;
  if (blockIdx.x == 0 && tid == 0) a.desc_table[a.slot] = a.desc;
  if (!a.vis) return;
  const int row0 = blockIdx.x * a.tile_rows;
  const int rows = min(a.tile_rows, a.desc.n_vis - row0);
  if (tid < rows) {
    const int v = row0 + tid;
    const int lp = v / a.page_tokens;
    const int off = v - lp * a.page_tokens;
    const uint64_t gva = reinterpret_cast<const uint64_t*>(a.meta + a.desc.page_off)[lp];
    const uint64_t pte = a.pte[(gva - a.gva_start) / a.page_bytes];
    s_dst[tid] = reinterpret_cast<uint8_t*>(pte & PTE_ADDR_MASK) + (size_t)off * a.row_bytes;
  }
  __syncthreads();
  // Source rows are contiguous; destinations come from the page walk.
  const int vpr = a.row_bytes >> 4;
  const int total = rows * vpr;
  const uint8_t* src = a.vis + (size_t)row0 * a.row_bytes;
  for (int e0 = tid; e0 < total; e0 += kBlock * U) {
    u32x4 v[U];
    int rr[U], cc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u * kBlock;
      rr[u] = e < total ? e / vpr : -1;
      cc[u] = e - (rr[u] < 0 ? 0 : rr[u]) * vpr;
      if (rr[u] >= 0) v[u] = load16(src + (size_t)e * 16);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (rr[u] >= 0) store16(s_dst[rr[u]] + (size_t)cc[u] * 16, v[u]);
  }
}

__global__ __launch_bounds__(kBlock) void k_cost(const SampleDesc* __restrict__ desc,
                                                  const int32_t* __restrict__ slots, int32_t n,
                                                  int64_t k, int64_t* __restrict__ out) {
  const int i = blockIdx.x * kBlock + threadIdx.x;
  if (i < n) {
    const int64_t l = desc[slots[i]].len;
    out[i] = k * l + l * l;
  }
}

constexpr int kUnroll = 8;

size_t pack_lds_bytes(const PackArgs& a) {
  return sizeof(PackSample) * (size_t)a.n + sizeof(int2) * (size_t)a.n_imgs +
         sizeof(void*) * (size_t)a.max_chunk_rows + sizeof(int32_t) * (size_t)(a.n + 1);
}

hipError_t launch_pack(const PackArgs& a, hipStream_t stream) {
  const int64_t vecs = (int64_t)a.n_tokens * (a.row_bytes >> 4);
  const int grid = vecs > 0 ? (int)((vecs + kChunkVecs - 1) / kChunkVecs) : 1;
  hipLaunchKernelGGL(k_pack, dim3(grid), dim3(kBlock), pack_lds_bytes(a), stream, a);
  return hipGetLastError();
}

hipError_t launch_write(const WriteArgs& a, hipStream_t stream) {
  const int rows = a.vis ? a.desc.n_vis : 0;
  const int grid = rows > 0 ? (rows + a.tile_rows - 1) / a.tile_rows : 1;
  hipLaunchKernelGGL(k_write<kUnroll>, dim3(grid), dim3(kBlock), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_cost(const SampleDesc* desc, const int32_t* slots, int32_t n, int64_t k,
                       int64_t* out_cost, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_cost, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0, stream, desc,
                     slots, n, k, out_cost);
  return hipGetLastError();
}

}  // namespace fp
