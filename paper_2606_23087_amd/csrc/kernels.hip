// HIP kernels of libflowpool for gfx950 (CDNA4).
//
// k_pack  : the consumer's translate-gather-pack of one microbatch
//           (paper Sec. 3.1 / Sec. 3.2): prefix sum of sample lengths ->
//           cu_seqlens; per row, the sample and its text/image segment; for
//           image rows the GVA page walk through the page table; then 16-byte
//           vector copies of every row from its page or embedding-table row
//           into the packed output, plus position ids.
// k_write : the producer's write of one sample's image rows into its pages,
//           through the same page table (Sec. 3.2 "write into the GVA
//           segment"), and publication of the sample descriptor.
// k_cost  : per-sample cost K*l + l^2 for the planner (Sec. 3.4).
//
// Nothing here is a dense contraction, so there is no MFMA: the pack is a
// bandwidth-bound gather whose cost is HBM bytes.

#include "fp_internal.h"

namespace fp {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load16(const uint8_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

__device__ __forceinline__ int32_t slot_at(const PackArgs& a, int i) {
  return a.slots_dev ? a.slots_dev[i] : a.slots_inline[i];
}

// Copies `rows` rows of `row_bytes` bytes: row r goes from src[r] to
// dst_base + r * row_bytes; a null src[r] skips the row. The rows x 16-byte
// vectors of the tile are spread evenly over the workgroup, U loads per
// thread in flight before their stores.
template <int U>
__device__ __forceinline__ void copy_tile(const uint8_t* const* src, uint8_t* dst_base, int rows,
                                          int row_bytes) {
  const int vpr = row_bytes >> 4;
  const int total = rows * vpr;
  for (int e0 = threadIdx.x; e0 < total; e0 += kBlock * U) {
    u32x4 v[U];
    int rr[U], cc[U];
    bool live[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + u * kBlock;
      live[u] = e < total;
      rr[u] = live[u] ? e / vpr : 0;
      cc[u] = e - rr[u] * vpr;
      const uint8_t* s = src[rr[u]];
      live[u] = live[u] && s != nullptr;
      if (live[u]) v[u] = load16(s + (size_t)cc[u] * 16);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (live[u]) store16(dst_base + (size_t)rr[u] * row_bytes + (size_t)cc[u] * 16, v[u]);
    }
  }
}

template <int U>
__global__ __launch_bounds__(kBlock) void k_pack(PackArgs a) {
  extern __shared__ int32_t s_cu[];                 // [n + 1]
  __shared__ const uint8_t* s_src[kMaxTileRows];
  __shared__ int32_t s_wsum[kBlock / 64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = a.n;

  // Exclusive prefix sum of the sample lengths, in plan order -> s_cu.
  if (tid == 0) s_cu[0] = 0;
  int carry = 0;
  for (int base = 0; base < n; base += kBlock) {
    const int i = base + tid;
    int v = (i < n) ? a.desc[slot_at(a, i)].len : 0;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(v, d, 64);
      if (lane >= d) v += t;
    }
    if (lane == 63) s_wsum[wave] = v;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kBlock / 64; ++w) {
      before += (w < wave) ? s_wsum[w] : 0;
      all += s_wsum[w];
    }
    if (i < n) s_cu[i + 1] = carry + before + v;
    carry += all;
    __syncthreads();
  }

  const bool write_meta = (a.tier_mask & 1) != 0;
  if (blockIdx.x == 0 && a.cu && write_meta) {
    for (int i = tid; i <= n; i += kBlock) a.cu[i] = s_cu[i];
  }

  const int row0 = blockIdx.x * a.tile_rows;
  const int rows = min(a.tile_rows, a.n_tokens - row0);

  // Resolve each row of the tile to its source address (one thread per row).
  if (tid < rows) {
    const int row = row0 + tid;
    int lo = 0, hi = n - 1;                          // last k with cu[k] <= row
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_cu[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const int r = row - s_cu[lo];
    const SampleDesc d = a.desc[slot_at(a, lo)];
    // Image j starts after img_pos[j] text rows and all earlier images' rows.
    const int2* img = reinterpret_cast<const int2*>(a.meta + d.img_off);
    int vis_before = 0;
    int vis_idx = -1;
    for (int j = 0; j < d.n_img; ++j) {
      const int2 pr = img[j];
      const int start = pr.x + vis_before;
      if (r < start) break;
      if (r < start + pr.y) { vis_idx = vis_before + (r - start); break; }
      vis_before += pr.y;
    }
    const uint8_t* src = nullptr;
    if (vis_idx < 0) {
      if (write_meta) {
        const int32_t id = reinterpret_cast<const int32_t*>(a.meta + d.text_off)[r - vis_before];
        src = a.table + (size_t)id * a.row_bytes;
      }
    } else {
      const int lp = vis_idx / a.page_tokens;
      const int off = vis_idx - lp * a.page_tokens;
      const uint64_t gva = reinterpret_cast<const uint64_t*>(a.meta + d.page_off)[lp];
      const uint64_t pte = a.pte[(gva - a.gva_start) / a.page_bytes];
      const int want = (pte & PTE_HOST) ? 2 : 1;
      if (a.tier_mask & want)
        src = reinterpret_cast<const uint8_t*>(pte & PTE_ADDR_MASK) + (size_t)off * a.row_bytes;
    }
    s_src[tid] = src;
    if (a.pos && write_meta) a.pos[row] = r;
  }
  __syncthreads();

  copy_tile<U>(s_src, a.out + (size_t)row0 * a.row_bytes, rows, a.row_bytes);
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

hipError_t launch_pack(const PackArgs& a, hipStream_t stream) {
  const int grid = a.n_tokens > 0 ? (a.n_tokens + a.tile_rows - 1) / a.tile_rows : 1;
  const size_t lds = sizeof(int32_t) * (size_t)(a.n + 1);
  hipLaunchKernelGGL(k_pack<kUnroll>, dim3(grid), dim3(kBlock), lds, stream, a);
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
