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

__device__ __forceinline__ u32x4 load16(const uint8_t* p) {
  return __builtin_nontemporal_load((g_u32x4_c*)p);
}

// Stores carry the nt and sc1 cache-policy bits of the gfx950 global store:
// on the pack this measured about 1.5 % faster than nt alone. The
// compiler has no builtin for that bit combination, hence the asm; it has
// no outputs, so the compiler still waits for the loaded data it stores.
__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1 nt" : : "v"(p), "v"(v) : "memory");
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

// Reads through constant-address-space views of uniform addresses compile to
// scalar loads (scalar cache), which do not queue behind the vector memory
// traffic of the copies.
typedef __attribute__((address_space(4))) const int32_t k_i32;
typedef __attribute__((address_space(4))) const int64_t k_i64;
typedef __attribute__((address_space(4))) const uint64_t k_u64;
typedef __attribute__((address_space(4))) const u32x4 k_u32x4;

// e / (row_bytes / 16) as a multiply and a shift (host-computed constants).
__device__ __forceinline__ int div_vpr(const PackArgs& a, int e) {
  return (int)(((uint64_t)(uint32_t)e * a.div_mul) >> a.div_shift);
}

// One workgroup packs one chunk of kChunkVecs 16-byte vectors of the output
// (rows are contiguous in the output, so a chunk is a contiguous byte range
// that may start and end inside rows): it finds, for every row the chunk
// touches, the row's sample (prefix sum of sample lengths) and segment, walks
// the page table for image rows, and then moves kVecsPerThread vectors per
// thread with all loads in flight before the stores.
//
// Headers passed by value and at most kWaveRows rows per wave (the usual
// case): each row is resolved by one wave with scalar loads, so the only
// vector memory loads are the copies. Otherwise the headers are staged in
// LDS and scanned there.
__global__ __launch_bounds__(kPackBlock) void k_pack(PackArgs a) {
  extern __shared__ __align__(16) uint8_t s_dyn[];
  __shared__ int32_t s_wsum[kPackBlock / 64];
  __shared__ int32_t s_skip[kPackBlock / 64];
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
  const int v0 = blockIdx.x * kChunkVecs;
  const int v1 = min(v0 + kChunkVecs, total);
  const int r0 = div_vpr(a, v0);
  const int rows = v1 > v0 ? div_vpr(a, v1 - 1) - r0 + 1 : 0;

  if (!a.samples_dev && rows <= kWaveRows * (kPackBlock / 64)) {
    // Each wave resolves rows wave, wave + 4, ... of the chunk on its own,
    // so the dependent load chains of different rows overlap. All of it is
    // wave-uniform and runs on scalar loads.
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (write_cu && tid == kPackBlock - 1) {
      int start = 0;
      for (int i = 0; i < a.n; ++i) {
        a.cu[i] = start;
        start += *(const k_i32*)(a.lens + i);
      }
      a.cu[a.n] = start;
    }
    for (int t = wave; t < rows; t += kPackBlock / 64) {
      const int row = r0 + t;
      // Sample k holding the row: running sum of the lengths, a group of
      // kLenGroup per scalar load (a short group ends the search sooner).
      int k = -1, start = 0;
      for (int b = 0; k < 0 && b < kInlineSamples; b += kLenGroup) {
        u32x4 g[kLenGroup / 4];
#pragma unroll
        for (int q = 0; q < kLenGroup / 4; ++q) g[q] = ((const k_u32x4*)(a.lens + b))[q];
#pragma unroll
        for (int q = 0; q < kLenGroup; ++q) {
          const int len = (int)g[q >> 2][q & 3];
          if (k < 0) {
            if (row < start + len) k = b + q;
            else start += len;
          }
        }
      }
      uint64_t src = 0;
      const int r = row - start;
      if (k >= 0) {
        const u32x4 h0 = ((const k_u32x4*)(a.samples + k))[0];
        const u32x4 h1 = ((const k_u32x4*)(a.samples + k))[1];
        const int n_img = (int)h0.y, img_base = (int)h0.z;
        const int64_t text_off = (int64_t)(((uint64_t)h1.y << 32) | h1.x);
        const int64_t page_off = (int64_t)(((uint64_t)h1.w << 32) | h1.z);
        // Segment of row r: image j starts after pos_j of the sample's text
        // rows and all rows of the images before it; text rows fill the gaps.
        int vis_before = 0, vidx = -1;
        bool done = false;
        for (int jb = 0; jb < n_img && !done; jb += kImgGroup) {
          const k_i32* pr = (const k_i32*)(a.imgs + img_base + jb);
          int pos_j[kImgGroup], ntok_j[kImgGroup];
#pragma unroll
          for (int j = 0; j < kImgGroup; ++j) {
            pos_j[j] = pr[2 * j];
            ntok_j[j] = pr[2 * j + 1];
          }
#pragma unroll
          for (int j = 0; j < kImgGroup; ++j) {
            if (!done && jb + j < n_img) {
              const int s0 = pos_j[j] + vis_before;
              if (r < s0) {
                done = true;
              } else if (r < s0 + ntok_j[j]) {
                vidx = vis_before + (r - s0);
                done = true;
              } else {
                vis_before += ntok_j[j];
              }
            }
          }
        }
        if (vidx < 0) {
          // Text row: its token id selects the embedding-table row.
          if (a.tier_mask & 1) {
            const int32_t id = *(const k_i32*)(a.meta + text_off + 4 * (int64_t)(r - vis_before));
            src = reinterpret_cast<uint64_t>(a.table) + (uint64_t)(uint32_t)id * (uint64_t)a.row_bytes;
          }
        } else {
          // Image row: page GVA from the sample's page list, page-table entry
          // from the GVA's page number, row inside the physical page.
          const int lp = (int)(((uint64_t)(uint32_t)vidx * a.pt_mul) >> a.pt_shift);
          const int off = vidx - lp * a.page_tokens;
          const uint64_t gva = *(const k_u64*)(a.meta + page_off + 8 * (int64_t)lp);
          const uint64_t vpn = __umul64hi(gva - a.gva_start, a.pb_mul) >> a.pb_shift;
          const uint64_t pte = *(const k_u64*)(a.pte + vpn);
          if (a.tier_mask & ((pte & PTE_HOST) ? 2 : 1))
            src = (pte & PTE_ADDR_MASK) + (uint64_t)off * (uint64_t)a.row_bytes;
        }
      }
      if (lane == 0) {
        s_src[t] = src;
        if (!src) my_skip = 1;
      }
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
      if (a.samples_dev && a.pos && write_meta && row * vpr >= v0) a.pos[row] = r;
    }
  }
  // One flag per wave, written before and read after the only barrier.
  const bool wave_skip = __any(my_skip);
  if ((tid & 63) == 0) s_skip[tid >> 6] = wave_skip ? 1 : 0;
  __syncthreads();
  int skip = 0;
#pragma unroll
  for (int w = 0; w < kPackBlock / 64; ++w) skip |= s_skip[w];

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
      const int row = div_vpr(a, e);
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

  // Position ids (headers passed by value): the last wave of workgroup b
  // writes the ids of rows [64 p, 64 p + 64) for blocks p = b, b + grid, ...,
  // so every cache line of them is written whole by one store instruction.
  // A lane's id is its row minus the first row of its sample, the largest
  // prefix sum of lengths not above the row.
  if (!a.samples_dev && a.pos && write_meta && tid >= kPackBlock - 64) {
    const int lane = tid & 63;
    for (int blk = blockIdx.x; blk * 64 < a.n_tokens; blk += gridDim.x) {
      const int row = blk * 64 + lane;
      const int last = min(blk * 64 + 63, a.n_tokens - 1);
      int start = 0, first = 0;
      for (int b = 0; b < kInlineSamples && start <= last; b += kLenGroup) {
        u32x4 g[kLenGroup / 4];
#pragma unroll
        for (int q = 0; q < kLenGroup / 4; ++q) g[q] = ((const k_u32x4*)(a.lens + b))[q];
#pragma unroll
        for (int q = 0; q < kLenGroup; ++q) {
          if (row >= start) first = start;
          start += (int)g[q >> 2][q & 3];
        }
      }
      if (row < a.n_tokens) a.pos[row] = row - first;
    }
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
