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
  for (int base = 0; base < n; base += kPackBlock) {
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
    for (int w = 0; w < kPackBlock / 64; ++w) {
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
// Page walk or text lookup of row r of a sample whose segment is already
// known: vis_idx >= 0 is the row's index among the sample's visual rows,
// otherwise text_idx is its index among the sample's text tokens.
__device__ __forceinline__ const uint8_t* row_source(const PackArgs& a, int64_t text_off,
                                                     int64_t page_off, int vis_idx, int text_idx) {
  if (vis_idx < 0) {
    if (!(a.tier_mask & 1)) return nullptr;
    const int32_t id = ld_global(reinterpret_cast<const int32_t*>(a.meta + text_off) + text_idx);
    return a.table + (size_t)id * a.row_bytes;
  }
  const int lp = vis_idx / a.page_tokens;
  const int off = vis_idx - lp * a.page_tokens;
  const uint64_t gva = ld_global(reinterpret_cast<const uint64_t*>(a.meta + page_off) + lp);
  const uint64_t pte = ld_global(a.pte + (gva - a.gva_start) / a.page_bytes);
  if (!(a.tier_mask & ((pte & PTE_HOST) ? 2 : 1))) return nullptr;
  return reinterpret_cast<const uint8_t*>(pte & PTE_ADDR_MASK) + (size_t)off * a.row_bytes;
}

// Reads through constant-address-space views of uniform addresses compile to
// scalar loads (scalar cache), which do not queue behind the vector memory
// traffic of the copies.
typedef __attribute__((address_space(4))) const int32_t k_i32;
typedef __attribute__((address_space(4))) const int64_t k_i64;
typedef __attribute__((address_space(4))) const uint64_t k_u64;

__device__ __forceinline__ int64_t readlane64(int64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), lane);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ PackSample ld_sample_scalar(const PackSample* p) {
  const k_i32* q = (const k_i32*)p;
  PackSample s;
  s.len = q[0];
  s.n_img = q[1];
  s.img_base = q[2];
  s.n_text = q[3];
  s.text_off = *(const k_i64*)(q + 4);
  s.page_off = *(const k_i64*)(q + 6);
  return s;
}

__device__ __forceinline__ int2 ld_pair_scalar(const int2* p) {
  const k_i32* q = (const k_i32*)p;
  int2 r;
  r.x = q[0];
  r.y = q[1];
  return r;
}

// One workgroup packs one chunk of kChunkVecs 16-byte vectors of the output
// (rows are contiguous in the output, so a chunk is a contiguous byte range
// that may start and end inside rows): it finds, for every row the chunk
// touches, the row's sample (prefix sum of sample lengths) and segment, walks
// the page table for image rows, and then moves kVecsPerThread vectors per
// thread with all loads in flight before the stores.
//
// Headers passed by value and at most kPackBlock rows per chunk (the usual case):
// the headers are read with scalar loads in one workgroup-uniform loop that
// also keeps the running prefix sum, so the only vector loads before the copy
// are the page walk and the text ids. Otherwise the headers are staged in LDS
// and scanned there.
__global__ __launch_bounds__(kPackBlock) void k_pack(PackArgs a) {
  extern __shared__ __align__(16) uint8_t s_dyn[];
  __shared__ int32_t s_wsum[kPackBlock / 64];
  PackSample* s_smp = reinterpret_cast<PackSample*>(s_dyn);
  int2* s_img = reinterpret_cast<int2*>(s_smp + a.n);
  uint64_t* s_src = reinterpret_cast<uint64_t*>(s_img + a.n_imgs);
  int32_t* s_cu = reinterpret_cast<int32_t*>(s_src + a.max_chunk_rows);
  const int tid = threadIdx.x;
  int my_skip = 0;                                  // a row of this chunk is not copied

  const bool write_meta = (a.tier_mask & 1) != 0;
  const bool write_cu = blockIdx.x == 0 && a.cu && write_meta;
  const int vpr = a.row_bytes >> 4;
  const int total = a.n_tokens * vpr;                 // the host keeps this below 2^31
  const int n_chunks = (total + kChunkVecs - 1) / kChunkVecs;
  const int v0 = blockIdx.x * kChunkVecs;
  const int v1 = min(v0 + kChunkVecs, total);
  const int r0 = v0 / vpr;
  const int rows = v1 > v0 ? (v1 - 1) / vpr - r0 + 1 : 0;

  if (!a.samples_dev && rows <= kPackBlock) {
    const bool own = tid < rows;
    const bool has_row = own;
    const int row = r0 + tid;
    const int owner_v0 = v0;
    int64_t text_off = 0, page_off = 0;
    int vis_idx = -1, text_idx = 0, r_in = 0;
    const int last_row = r0 + rows - 1;
    int start = 0;                                   // first row of sample i (uniform)
    for (int i = 0; i < a.n; ++i) {
      const PackSample sp = ld_sample_scalar(a.samples + i);
      if (write_cu && tid == 0) a.cu[i] = start;
      const bool mine = has_row && row >= start && row < start + sp.len;
      if (__any(mine)) {
        // Image j starts after pr.x of the sample's text rows and all rows of
        // the images before it; text rows fill the gaps.
        const int r = row - start;
        int vis_before = 0, vidx = -1;
        bool found = false;
        for (int j = 0; j < sp.n_img; ++j) {
          const int2 pr = ld_pair_scalar(a.imgs + sp.img_base + j);
          if (!found) {
            const int s0 = pr.x + vis_before;
            if (r < s0) {
              found = true;
            } else if (r < s0 + pr.y) {
              vidx = vis_before + (r - s0);
              found = true;
            } else {
              vis_before += pr.y;
            }
          }
        }
        if (mine) {
          r_in = r;
          vis_idx = vidx;
          text_idx = r - vis_before;
          text_off = sp.text_off;
          page_off = sp.page_off;
        }
      }
      start += sp.len;
      if (!write_cu && start > last_row) break;
    }
    if (write_cu && tid == 0) a.cu[a.n] = start;
    if (rows <= 64) {
      // Wave 0 walks the rows one after another with scalar loads; rows on
      // the same page reuse the previous translation.
      if (tid < 64) {
        uint64_t my_src = 0;
        int64_t prev_page = -1;
        uint64_t prev_base = 0;
        for (int t = 0; t < rows; ++t) {
          const int vis = __builtin_amdgcn_readlane(vis_idx, t);
          uint64_t src = 0;
          if (vis < 0) {
            if (a.tier_mask & 1) {
              const int tix = __builtin_amdgcn_readlane(text_idx, t);
              const int64_t toff = readlane64(text_off, t);
              const int32_t id = *(const k_i32*)(a.meta + toff + 4 * (int64_t)tix);
              src = reinterpret_cast<uint64_t>(a.table) + (uint64_t)id * (uint64_t)a.row_bytes;
            }
          } else {
            const int64_t poff = readlane64(page_off, t);
            const int lp = vis / a.page_tokens;
            const int off = vis - lp * a.page_tokens;
            const int64_t page_key = poff + 8 * (int64_t)lp;   // position of the page's GVA
            if (page_key != prev_page) {
              const uint64_t gva = *(const k_u64*)(a.meta + page_key);
              const uint64_t pte = *(const k_u64*)(a.pte + (gva - a.gva_start) / a.page_bytes);
              prev_base = (a.tier_mask & ((pte & PTE_HOST) ? 2 : 1)) ? (pte & PTE_ADDR_MASK) : 0;
              prev_page = page_key;
            }
            src = prev_base ? prev_base + (uint64_t)off * (uint64_t)a.row_bytes : 0;
          }
          if (tid == t) my_src = src;
        }
        if (has_row) {
          s_src[tid] = my_src;
          if (!my_src) my_skip = 1;
          if (a.pos && write_meta && row * vpr >= owner_v0) a.pos[row] = r_in;
        }
      }
    } else if (has_row) {
      const uint8_t* src = row_source(a, text_off, page_off, vis_idx, text_idx);
      s_src[tid] = reinterpret_cast<uint64_t>(src);
      if (own && !src) my_skip = 1;
      if (a.pos && write_meta && row * vpr >= owner_v0) a.pos[row] = r_in;
    }
  } else {
    const PackSample* gs = a.samples_dev ? a.samples_dev : a.samples;
    const int2* gi = a.imgs_dev ? a.imgs_dev : a.imgs;
    for (int i = tid; i < a.n; i += kPackBlock) s_smp[i] = ld_sample(gs + i);
    for (int i = tid; i < a.n_imgs; i += kPackBlock) s_img[i] = ld_pair(gi + i);
    __syncthreads();
    block_scan_lengths(s_smp, a.n, s_cu, s_wsum);
    if (write_cu) {
      for (int i = tid; i <= a.n; i += kPackBlock) a.cu[i] = s_cu[i];
    }
    for (int t = tid; t < rows; t += kPackBlock) {
      const int row = r0 + t;
      const int k = sample_of(s_cu, a.n, row);
      const int r = row - s_cu[k];
      const uint8_t* src = resolve_row(a, s_smp[k], s_img, r);
      s_src[t] = reinterpret_cast<uint64_t>(src);
      if (!src) my_skip = 1;
      if (a.pos && write_meta && row * vpr >= v0) a.pos[row] = r;
    }
  }
  const bool skip = __syncthreads_or(my_skip);

  // Vector e of the chunk belongs to row e / vpr (multiply-shift division).
  // A vector is live if it lies in the chunk and its row is copied; only
  // live vectors get an address, dead ones are never loaded or stored.
  uint64_t from[kVecsPerThread];
  bool live[kVecsPerThread];
#pragma unroll
  for (int u = 0; u < kVecsPerThread; ++u) {
    const int e = v0 + u * kPackBlock + tid;
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
  if (v1 - v0 == kChunkVecs && !skip) {
    // Whole chunk, every row copied: no predication, so the compiler can keep
    // all loads in flight and wait for them one at a time before each store.
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u) v[u] = load16(reinterpret_cast<const uint8_t*>(from[u]));
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      store16(a.out + (size_t)(v0 + u * kPackBlock + tid) * 16, v[u]);
  } else {
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      if (live[u]) v[u] = load16(reinterpret_cast<const uint8_t*>(from[u]));
#pragma unroll
    for (int u = 0; u < kVecsPerThread; ++u)
      if (live[u]) store16(a.out + (size_t)(v0 + u * kPackBlock + tid) * 16, v[u]);
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
  hipLaunchKernelGGL(k_pack, dim3(grid), dim3(kPackBlock), pack_lds_bytes(a), stream, a);
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
