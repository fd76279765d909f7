// HIP kernels of libflowpool for gfx950 (CDNA4).
//
// k_pack  : the consumer's translate-gather-pack of one microbatch
//           (paper Sec. 3.1 / Sec. 3.2): per row, its run (a stretch of one
//           sample's text rows or image rows, listed by the host in row
//           order); for image rows the GVA page walk through the page table;
//           then 16-byte vector copies of every row from its page or
//           embedding-table row into the packed output; cu_seqlens as a
//           wave-wide prefix sum of the sample lengths, and position ids.
// k_write : the producer's write of one sample's image rows into its pages,
//           through the same page table (Sec. 3.2, producer side), and
//           publication of the sample descriptor.
// k_cost  : per-sample cost K*l + l^2 for the planner (Sec. 3.4).
//
// Nothing here is a dense contraction, so there is no MFMA: the pack is a
// bandwidth-bound gather whose cost is HBM bytes.

#include "fp_internal.h"

#include <algorithm>
#include <cstring>

namespace fp {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// Global-address-space views: loads through them compile to global_load
// (vector memory counter only) instead of flat loads, which also count
// against the LDS counter and force the compiler to wait for each one.
typedef __attribute__((address_space(1))) const u32x4 g_u32x4_c;

__device__ __forceinline__ u32x4 load16(const uint8_t* p) {
  return __builtin_nontemporal_load((g_u32x4_c*)p);
}

// Embedding-table rows are read at random ids, a few KiB each, and may be
// read again by later packs: plain loads let the memory-side cache keep
// them (see kTablePlainLoads), while rows read in page order are about 2 %
// faster non-temporal. The policy is an instruction bit, so the pack picks
// it per chunk.
__device__ __forceinline__ u32x4 load16_table(const uint8_t* p) {
  return *(g_u32x4_c*)p;
}

// Stores carry the nt and sc1 cache-policy bits of the gfx950 global store:
// on the pack this measured about 1.5 % faster than nt alone. The
// compiler has no builtin for that bit combination, hence the asm; it has
// no outputs, so the compiler still waits for the loaded data it stores.
// The compiler does not see inside the asm, so the asm carries the wait that
// gfx940-class parts need between a store of more than 8 bytes and a VALU
// write to its data registers (two wait states): without it the compiler
// may reuse those registers right after the store and corrupt its data.
__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1 nt\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
}

// Reads through constant-address-space views of uniform addresses compile to
// scalar loads (scalar cache), which do not queue behind the vector memory
// traffic of the copies; the per-lane path reads through global views.
// Loads for the two ways rows are resolved: kScalar (one row per wave,
// wave-uniform addresses) or per lane.
template <bool kScalar, typename T>
__device__ __forceinline__ T ld(const void* p) {
  if constexpr (kScalar) {
    return *(const __attribute__((address_space(4))) T*)p;
  } else {
    return *(const __attribute__((address_space(1))) T*)p;
  }
}

// The pack's leading kernel arguments: everything a wave needs to address its
// row's bucket run and bucket-index entry. They are separate scalar arguments, ahead of PackArgs,
// so that the hardware preloads them into scalar registers at wave launch
// (kernarg preloading); the first loads of the row lookup then leave at once,
// alongside the kernel-argument loads of the rest.
struct PackHead {
  int32_t g0, g1, t1, t2;   // chunk geometry (as in PackPlan)
  uint64_t div_mul;         // e / (row_bytes / 16) == (e * div_mul) >> div_shift
  int32_t div_shift;
  int32_t bucket_shift;
  const uint8_t* tb;        // run table: staged copy, or null = the one in PackArgs
  int32_t off_brun;         // byte offsets of the bucket runs and the bucket index in the run table
  int32_t off_bucket;
  int32_t total;            // vectors of the microbatch
};

// A run index: bucket size and where its bucket runs and bucket entries sit
// in the run table.
struct RunIndex {
  int32_t shift, off_brun, off_bucket;
};

// e / (row_bytes / 16) as a multiply and a shift (host-computed constants).
__device__ __forceinline__ int div_vpr(const PackHead& h, int e) {
  return (int)(((uint64_t)(uint32_t)e * h.div_mul) >> h.div_shift);
}

// One run, as a single 16-byte load.
template <bool kScalar>
__device__ __forceinline__ PackRun ld_run(const PackRun* rp) {
  const u32x4 d = ld<kScalar, u32x4>(rp);
  return PackRun{(int32_t)d.x, (int32_t)d.y, (int32_t)d.z, (int32_t)d.w};
}

// The first two loads of a row's lookup, independent of each other: its
// bucket's run (the run holding the bucket's first row) and the word of the
// bucket index that holds that run's number.
struct BucketHit {
  PackRun r;
  uint32_t w;
};

template <bool kScalar>
__device__ __forceinline__ BucketHit bucket_of(const RunIndex& x, const uint8_t* tb, int row) {
  const int b = row >> x.shift;
  return BucketHit{ld_run<kScalar>(reinterpret_cast<const PackRun*>(tb + x.off_brun) + b),
                   ld<kScalar, uint32_t>(tb + x.off_bucket + 4 * (b >> 1))};
}

// Run holding row `row`: its bucket's run, or a later one, stepped to from
// that run's number when the bucket's run ends at or before the row.
template <bool kScalar>
__device__ __forceinline__ PackRun run_of(const RunIndex& x, int32_t off_runs, const uint8_t* tb, int row,
                                          const BucketHit& hit, int* s_out = nullptr) {
  PackRun r = hit.r;
  if (r.end <= row || s_out) {
    const int b = row >> x.shift;
    int s = (int)((b & 1) ? (hit.w >> 16) : (hit.w & 0xffffu));
    const PackRun* runs = reinterpret_cast<const PackRun*>(tb + off_runs);
    while (r.end <= row) r = ld_run<kScalar>(runs + ++s);
    if (s_out) *s_out = s;
  }
  return r;
}

// Row of physical memory holding visual row `vidx` of an image run: visual
// index -> page GVA -> page-table entry (the GVA's page number) -> row in the
// physical page. `word` >= 0: the sample's page GVAs start at 64-bit word
// `word` of the arena (the page list). `word` < 0: the sample's pages have
// consecutive GVAs, page lp's GVA is page 0's plus lp pages, and -word - 1 is
// page 0's page number, so the page number needs no load. Returns the
// page-table entry's flags in *flags.
template <bool kScalar, class Args>
__device__ __forceinline__ uint64_t walk(const Args& a, int32_t word, uint32_t vidx, uint64_t* flags) {
  const int lp = (int)(((uint64_t)vidx * a.pt_mul) >> a.pt_shift);
  const int in_page = (int)vidx - lp * a.page_tokens;
  uint64_t vpn;
  if (word < 0) {
    vpn = (uint64_t)(-(int64_t)word - 1) + (uint64_t)lp;
  } else {
    const uint64_t gva = ld<kScalar, uint64_t>(a.meta + 8 * ((int64_t)word + lp));
    vpn = __umul64hi(gva - a.gva_start, a.pb_mul) >> a.pb_shift;
  }
  const uint64_t pte = ld<kScalar, uint64_t>(a.pte + vpn);
  *flags = pte;
  return (pte & PTE_ADDR_MASK) + (uint64_t)in_page * (uint64_t)a.row_bytes;
}

template <class Args>
__device__ __forceinline__ uint64_t text_row(const Args& a, int32_t id) {
  return reinterpret_cast<uint64_t>(a.table) + (uint64_t)(uint32_t)id * (uint64_t)a.row_bytes;
}

// Source address of packed row `row` of run r, or 0 when the tier mask
// leaves the row out. A text row's id selects an embedding-table row; an
// image row walks the page table.
template <bool kScalar, class Args>
__device__ __forceinline__ uint64_t row_source(const Args& a, const PackRun& run, int row) {
  if (run.head < 0) {
    if (!(a.tier_mask & 1)) return 0;
    return text_row(a, ld<kScalar, int32_t>(a.meta + 4 * ((int64_t)run.word + row)));
  }
  uint64_t flags = 0;
  const uint64_t src = walk<kScalar>(a, run.word, (uint32_t)(row + run.vdelta), &flags);
  if (!(a.tier_mask & ((flags & PTE_HOST) ? 2 : 1))) return 0;
  return src;
}

// Moves a thread's first N vectors of a chunk: vector u comes from from[u] and
// goes to vector v0 + u * kPackBlock + tid of the output. kWhole: every
// vector is live, so there is no predication and the compiler keeps all
// loads in flight and waits for them one at a time before each store;
// otherwise only live vectors are loaded and stored. kTable: the chunk holds
// embedding-table rows and takes plain loads, else non-temporal ones. The
// two load forms differ only in a cache-policy bit, which the compiler drops
// when it merges otherwise identical code of two branches into one; the
// table form is therefore fenced by asm statements (they emit no
// instructions) that nothing can be merged across.
template <int N, bool kTable, bool kWhole>
__device__ __forceinline__ void copy_vectors(const uint64_t* from, const bool* live, uint8_t* out, int v0,
                                             int tid) {
  if constexpr (kTable) asm volatile(";; table-row chunk");
  u32x4 v[N];
#pragma unroll
  for (int u = 0; u < N; ++u)
    if (kWhole || live[u]) {
      const uint8_t* p = reinterpret_cast<const uint8_t*>(from[u]);
      v[u] = kTable ? load16_table(p) : load16(p);
    }
#pragma unroll
  for (int u = 0; u < N; ++u)
    if (kWhole || live[u]) store16(out + (size_t)(v0 + u * kPackBlock + tid) * 16, v[u]);
  if constexpr (kTable) asm volatile(";; table-row chunk end");
}

// One workgroup packs one chunk of 256 * VPT 16-byte vectors of the output
// (rows are contiguous in the output, so a chunk is a contiguous byte range
// that may start and end inside rows; the last chunks are smaller): it
// resolves the source of every row the chunk touches, then moves up to VPT
// vectors per thread with all loads in flight before the stores. VPT is 3
// (12 KiB chunks), or 2 for rows of kSmallChunkRowBytes or more.
//
// Up to kWaveRows rows per wave (the usual case: a chunk touches two or three
// rows at realistic hidden sizes), each row is resolved by one wave with
// scalar loads, so the only vector memory loads are the copies. Chunks of
// many short rows resolve one row per lane.
template <int VPT, class Args>
__global__ __launch_bounds__(kPackBlock) void k_pack(int32_t g0, int32_t g1, int32_t t1, int32_t t2,
                                                      uint64_t div_mul, int32_t div_shift, int32_t bucket_shift,
                                                      const uint8_t* staged, int32_t off_brun, int32_t off_bucket,
                                                      int32_t total, Args a) {
  constexpr int kChunk = kPackBlock * VPT;       // vectors of a full chunk
  extern __shared__ __align__(16) uint64_t s_src[];
  __shared__ int32_t s_flags[kPackBlock / 64];
  const PackHead h{g0, g1, t1, t2, div_mul, div_shift, bucket_shift, staged, off_brun, off_bucket, total};
  const RunIndex cx{h.bucket_shift, h.off_brun, h.off_bucket};
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const uint8_t* tb = h.tb ? h.tb : reinterpret_cast<const uint8_t*>(a.lens);
  int my_skip = 0;                                  // a row of this chunk is not copied
  int my_table = 0;                                 // a row of this chunk is an embedding-table row

  const int bx = (int)blockIdx.x;
  int v0, v1;
  if (bx < h.g0) {
    v0 = bx * kChunk;
    v1 = v0 + kChunk;
  } else if (bx < h.g1) {
    v0 = h.t1 + (bx - h.g0) * kTail1Vecs;
    v1 = min(v0 + kTail1Vecs, h.t2);
  } else {
    v0 = h.t2 + (bx - h.g1) * kTail2Vecs;
    v1 = min(v0 + kTail2Vecs, h.total);
  }
  const int r0 = div_vpr(h, v0);
  const int rows = v1 > v0 ? div_vpr(h, v1 - 1) - r0 + 1 : 0;
  // The bucket run and index entry of the wave's first row (a row of the
  // chunk; row 0 of an empty pack, whose table always has them), then the other kernel
  // arguments the row resolution uses in one batch of scalar loads, in flight
  // together with it (the compiler would otherwise split the batch and load
  // it first).
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const BucketHit w0 = bucket_of<true>(cx, tb, r0 + min(wave, max(rows - 1, 0)));
  asm volatile("" : : "s"(w0.w), "s"(w0.r.end), "s"(w0.r.head), "s"(w0.r.vdelta), "s"(w0.r.word),
               "s"(a.off_runs), "s"(a.meta), "s"(a.table), "s"(a.pte), "s"(a.gva_start), "s"(a.pt_mul), "s"(a.pt_shift), "s"(a.pb_mul), "s"(a.pb_shift), "s"(a.page_tokens),
               "s"(a.tier_mask), "s"(a.row_bytes));
  const bool write_meta = (a.tier_mask & 1) != 0;
  const int vpr = a.row_bytes >> 4;

  if (rows <= kWaveRows * (kPackBlock / 64)) {
    // Wave w resolves rows w, w + 4, ... of the chunk, so the dependent load
    // chains of different rows overlap.
    for (int t = wave; t < rows; t += kPackBlock / 64) {
      const int row = r0 + t;
      const BucketHit w = t == wave ? w0 : bucket_of<true>(cx, tb, row);
      const PackRun run = run_of<true>(cx, a.off_runs, tb, row, w);
      const uint64_t src = row_source<true>(a, run, row);
      if (lane == 0) {
        s_src[t] = src;
        if (!src) my_skip = 1;
        else if (run.head < 0) my_table = 1;
      }
    }
  } else {
    for (int t = tid; t < rows; t += kPackBlock) {
      const int row = r0 + t;
      const PackRun run = run_of<false>(cx, a.off_runs, tb, row, bucket_of<false>(cx, tb, row));
      const uint64_t src = row_source<false>(a, run, row);
      s_src[t] = src;
      if (!src) my_skip = 1;
      else if (run.head < 0) my_table = 1;
    }
  }
  // Flags per wave, written before and read after the only barrier.
  const int wave_flags = (__any(my_skip) ? 1 : 0) | (__any(my_table) ? 2 : 0);
  if (lane == 0) s_flags[tid >> 6] = wave_flags;
  __syncthreads();
  int flags = 0;
#pragma unroll
  for (int w = 0; w < kPackBlock / 64; ++w) flags |= s_flags[w];
  flags = __builtin_amdgcn_readfirstlane(flags);   // the same in every lane
  const bool skip = (flags & 1) != 0;
  // Plain loads for the whole chunk (for tables small enough to cache).
  const bool table = (flags & 2) != 0 && (a.tier_mask & kTablePlainLoads) != 0;

  // Vector e of the chunk belongs to row e / vpr (multiply-shift division).
  // A vector is live if it lies in the chunk and its row is copied; only
  // live vectors get an address, dead ones are never loaded or stored.
  uint64_t from[VPT];
  bool live[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int e = v0 + u * kPackBlock + tid;
    from[u] = 0;
    live[u] = false;
    if (e < v1) {
      const int row = div_vpr(h, e);
      const uint64_t base = s_src[row - r0];
      live[u] = base != 0;
      from[u] = live[u] ? base + (uint64_t)(e - row * vpr) * 16 : 0;
    }
  }
  // Full chunks and the two tail sizes (whole multiples of the block) with
  // every row copied move their vectors unpredicated; the last chunk and
  // chunks with rows the tier mask leaves out are predicated per vector.
  static_assert(kTail1Vecs % kPackBlock == 0 && kTail2Vecs % kPackBlock == 0 && kTail2Vecs < kTail1Vecs &&
                    kTail1Vecs <= kChunk, "tail chunks are whole multiples of the block");
  constexpr int kT1 = kTail1Vecs / kPackBlock, kT2 = kTail2Vecs / kPackBlock;
  const int n_vec = v1 - v0;
  if (!skip && n_vec == kChunk) {
    if (table) copy_vectors<VPT, true, true>(from, live, a.out, v0, tid);
    else copy_vectors<VPT, false, true>(from, live, a.out, v0, tid);
  } else if (!skip && n_vec == kTail1Vecs) {
    if (table) copy_vectors<kT1, true, true>(from, live, a.out, v0, tid);
    else copy_vectors<kT1, false, true>(from, live, a.out, v0, tid);
  } else if (!skip && n_vec == kTail2Vecs) {
    if (table) copy_vectors<kT2, true, true>(from, live, a.out, v0, tid);
    else copy_vectors<kT2, false, true>(from, live, a.out, v0, tid);
  } else {
    if (table) copy_vectors<VPT, true, false>(from, live, a.out, v0, tid);
    else copy_vectors<VPT, false, false>(from, live, a.out, v0, tid);
  }

  // cu_seqlens and position ids, by the last wave after its copies.
  // Workgroup 0 writes cu_seqlens: an exclusive prefix sum of the sample
  // lengths, 64 samples per step of a wave-wide scan. Workgroup b writes the
  // position ids of rows [64 p, 64 p + 64) for blocks p = b, b + grid, ...,
  // so every cache line of them is written whole by one store instruction:
  // a row's id is the row minus the first row of its sample, taken from the
  // runs that start inside the block.
  if (write_meta && tid >= kPackBlock - 64) {
    if (blockIdx.x == 0 && a.cu) {
      if (lane == 0) a.cu[0] = 0;
      int carry = 0;
      for (int base = 0; base < a.n; base += 64) {
        const int i = base + lane;
        int v = i < a.n ? ld<false, int32_t>(tb + 4 * i) : 0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int t = __shfl_up(v, d, 64);
          if (lane >= d) v += t;
        }
        if (i < a.n) a.cu[i + 1] = carry + v;
        carry += __shfl(v, 63, 64);
      }
    }
    if (a.pos) {
      const PackRun* runs = reinterpret_cast<const PackRun*>(tb + a.off_runs);
      for (int blk = blockIdx.x; blk * 64 < a.n_tokens; blk += gridDim.x) {
        const int first = blk * 64, row = first + lane;
        const int last = min(first + 63, a.n_tokens - 1);
        int s;
        PackRun r = run_of<true>(cx, a.off_runs, tb, first, bucket_of<true>(cx, tb, first), &s);
        int start = r.head & 0x7fffffff;
        while (r.end <= last) {
          const int next = r.end;
          r = ld_run<true>(runs + ++s);
          if (row >= next) start = r.head & 0x7fffffff;
        }
        if (row < a.n_tokens) a.pos[row] = row - start;
      }
    }
  }
}

// Producer write (Sec. 3.2): the sample's contiguous visual rows are cut into
// chunks of kChunkVecs vectors; each workgroup loops over chunks b, b + grid,
// ... (the grid is capped at kWriteGrid). Per chunk, each wave walks the page
// table for rows wave, wave + 4, ... with scalar loads (visual row -> page
// GVA -> page-table entry -> row in the physical page), a barrier shares the
// destinations, and every thread moves up to kVecsPerThread vectors. Chunks
// of many short rows walk one row per lane. Workgroup 0 also publishes the
// sample descriptor.
__global__ __launch_bounds__(kPackBlock) void k_write(WriteArgs a) {
  extern __shared__ __align__(16) uint64_t s_dst[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  if (blockIdx.x == 0 && tid == 0) a.desc_table[a.slot] = a.desc;
  if (!a.vis) return;
  const int vpr = a.row_bytes >> 4;
  const int total = a.desc.n_vis * vpr;               // the host keeps this below 2^31
  const uint64_t* pages = reinterpret_cast<const uint64_t*>(a.meta + a.desc.page_off);
  auto div_row = [&](int e) { return (int)(((uint64_t)(uint32_t)e * a.dv.div_mul) >> a.dv.div_shift); };
  auto dest = [&](auto ldk, int v) {
    const int lp = (int)(((uint64_t)(uint32_t)v * a.dv.pt_mul) >> a.dv.pt_shift);
    const int in_page = v - lp * a.page_tokens;
    const uint64_t gva = ldk(pages + lp);
    const uint64_t vpn = __umul64hi(gva - a.gva_start, a.dv.pb_mul) >> a.dv.pb_shift;
    return (ldk(a.pte + vpn) & PTE_ADDR_MASK) + (uint64_t)in_page * (uint64_t)a.row_bytes;
  };
  for (int64_t chunk = blockIdx.x; chunk * kChunkVecs < total; chunk += gridDim.x) {
    const int v0 = (int)chunk * kChunkVecs;
    const int v1 = min(v0 + kChunkVecs, total);
    const int r0 = div_row(v0);
    const int rows = div_row(v1 - 1) - r0 + 1;
    if (rows <= kWaveRows * (kPackBlock / 64)) {
      const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
      for (int t = wave; t < rows; t += kPackBlock / 64) {
        const uint64_t d = dest([](const uint64_t* p) { return ld<true, uint64_t>(p); }, r0 + t);
        if (lane == 0) s_dst[t] = d;
      }
    } else {
      for (int t = tid; t < rows; t += kPackBlock)
        s_dst[t] = dest([](const uint64_t* p) { return ld<false, uint64_t>(p); }, r0 + t);
    }
    __syncthreads();
    uint64_t to[kVecsPerThread];
    u32x4 v[kVecsPerThread];
    if (v1 - v0 == kChunkVecs) {
#pragma unroll
      for (int u = 0; u < kVecsPerThread; ++u) {
        const int e = v0 + u * kPackBlock + tid;
        const int row = div_row(e);
        to[u] = s_dst[row - r0] + (uint64_t)(e - row * vpr) * 16;
        v[u] = load16(a.vis + (size_t)e * 16);
      }
#pragma unroll
      for (int u = 0; u < kVecsPerThread; ++u) store16(reinterpret_cast<uint8_t*>(to[u]), v[u]);
    } else {
#pragma unroll
      for (int u = 0; u < kVecsPerThread; ++u) {
        const int e = v0 + u * kPackBlock + tid;
        if (e < v1) {
          const int row = div_row(e);
          to[u] = s_dst[row - r0] + (uint64_t)(e - row * vpr) * 16;
          v[u] = load16(a.vis + (size_t)e * 16);
        }
      }
#pragma unroll
      for (int u = 0; u < kVecsPerThread; ++u)
        if (v0 + u * kPackBlock + tid < v1) store16(reinterpret_cast<uint8_t*>(to[u]), v[u]);
    }
    __syncthreads();                                  // s_dst is rewritten for the next chunk
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

size_t pack_lds_bytes(const PackPlan& pl) { return sizeof(uint64_t) * (size_t)std::max(pl.max_chunk_rows, 1); }

// Chunk geometry over `vecs` vectors: full chunks of kPackBlock * vpt
// vectors, then a wave of resident workgroups (CUs x kPackPerCU) of
// kTail1Vecs, then half a wave of kTail2Vecs.
static void chunk_geometry(int64_t vecs, int n_cu, PackPlan* pl) {
  const int64_t chunk = (int64_t)kPackBlock * pl->vpt;
  const int64_t wave = (int64_t)std::max(n_cu, 1) * kPackPerCU;
  const int64_t t2 = std::max<int64_t>(vecs - (wave / 2) * kTail2Vecs, 0);
  const int64_t t1 = (std::max<int64_t>(t2 - wave * kTail1Vecs, 0) / chunk) * chunk;
  pl->g0 = (int32_t)(t1 / chunk);
  pl->g1 = (int32_t)(pl->g0 + (t2 - t1 + kTail1Vecs - 1) / kTail1Vecs);
  pl->t1 = (int32_t)t1;
  pl->t2 = (int32_t)t2;
}

static int vectors_per_thread(int64_t row_bytes) { return row_bytes >= kSmallChunkRowBytes ? 2 : kVecsPerThread; }

void pack_chunks(PackPlan* pl, int n_cu) {
  pl->vpt = vectors_per_thread(pl->a.row_bytes);
  chunk_geometry((int64_t)pl->a.n_tokens * (pl->a.row_bytes >> 4), n_cu, pl);
}

// The compact arguments of a small pack: the same scalar fields, the table
// copied into the smaller arrays, offsets relative to them.
static void small_args(const PackPlan& pl, PackArgsSmall* s) {
  std::memcpy(static_cast<void*>(s), &pl.a, offsetof(PackArgs, lens));
  std::memcpy(s->lens, pl.a.lens, sizeof(int32_t) * (size_t)pl.a.n);
  std::memcpy(s->runs, pl.a.runs, sizeof(PackRun) * (size_t)pl.n_runs);
  std::memcpy(s->brun, pl.a.brun, sizeof(PackRun) * (size_t)pl.n_buckets);
  std::memcpy(s->bucket, pl.a.bucket, sizeof(uint16_t) * (size_t)pl.n_buckets);
  s->off_runs = (int32_t)(offsetof(PackArgsSmall, runs) - offsetof(PackArgsSmall, lens));
  s->off_brun = (int32_t)(offsetof(PackArgsSmall, brun) - offsetof(PackArgsSmall, lens));
  s->off_bucket = (int32_t)(offsetof(PackArgsSmall, bucket) - offsetof(PackArgsSmall, lens));
}

template <int VPT, class Args>
static void launch_pack_as(const PackPlan& pl, const Args& a, int grid, int32_t total, hipStream_t stream) {
  hipLaunchKernelGGL((k_pack<VPT, Args>), dim3(grid), dim3(kPackBlock), pack_lds_bytes(pl), stream, pl.g0, pl.g1,
                     pl.t1, pl.t2, pl.div_mul, pl.div_shift, a.bucket_shift, pl.staged, a.off_brun, a.off_bucket,
                     total, a);
}

hipError_t launch_pack(const PackPlan& pl, hipStream_t stream) {
  const int64_t vecs = (int64_t)pl.a.n_tokens * (pl.a.row_bytes >> 4);
  const int64_t grid64 = pl.g1 + (vecs - pl.t2 + kTail2Vecs - 1) / kTail2Vecs;
  const int grid = grid64 > 0 ? (int)grid64 : 1;
  const int32_t total = (int32_t)vecs;               // the host keeps this below 2^31
  if (pl.small) {
    PackArgsSmall s{};
    small_args(pl, &s);
    if (pl.vpt == 2) launch_pack_as<2>(pl, s, grid, total, stream);
    else launch_pack_as<kVecsPerThread>(pl, s, grid, total, stream);
  } else {
    if (pl.vpt == 2) launch_pack_as<2>(pl, pl.a, grid, total, stream);
    else launch_pack_as<kVecsPerThread>(pl, pl.a, grid, total, stream);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Measurement aids, not steps of the method: a plain copy, and a plain gather
// of rows from given addresses into consecutive output rows, with the pack's
// chunk geometry (chunks of 256 threads x VPT vectors, the same shrinking
// tail stages) and its load and store cache policy. They move the bytes a
// pack moves and do nothing else, so the pack can be timed against them in
// the same run.

template <int VPT>
__device__ __forceinline__ void chunk_range(int32_t g0, int32_t g1, int32_t t1, int32_t t2, int32_t total, int* v0,
                                            int* v1) {
  constexpr int kChunk = kPackBlock * VPT;
  const int bx = (int)blockIdx.x;
  if (bx < g0) {
    *v0 = bx * kChunk;
    *v1 = *v0 + kChunk;
  } else if (bx < g1) {
    *v0 = t1 + (bx - g0) * kTail1Vecs;
    *v1 = min(*v0 + kTail1Vecs, t2);
  } else {
    *v0 = t2 + (bx - g1) * kTail2Vecs;
    *v1 = min(*v0 + kTail2Vecs, total);
  }
}

// The pack's copy of one chunk's vectors (see k_pack): full chunks and the
// two tail sizes unpredicated, the last chunk predicated per vector.
template <int VPT, bool kTable>
__device__ __forceinline__ void copy_chunk(const uint64_t* from, const bool* live, uint8_t* dst, int v0, int v1) {
  constexpr int kT1 = kTail1Vecs / kPackBlock, kT2 = kTail2Vecs / kPackBlock;
  const int tid = (int)threadIdx.x;
  if (v1 - v0 == kPackBlock * VPT) copy_vectors<VPT, kTable, true>(from, live, dst, v0, tid);
  else if (v1 - v0 == kTail1Vecs) copy_vectors<kT1, kTable, true>(from, live, dst, v0, tid);
  else if (v1 - v0 == kTail2Vecs) copy_vectors<kT2, kTable, true>(from, live, dst, v0, tid);
  else copy_vectors<VPT, kTable, false>(from, live, dst, v0, tid);
}

template <int VPT>
__global__ __launch_bounds__(kPackBlock) void k_copy(int32_t g0, int32_t g1, int32_t t1, int32_t t2, int32_t total,
                                                      const uint8_t* src, uint8_t* dst) {
  int v0, v1;
  chunk_range<VPT>(g0, g1, t1, t2, total, &v0, &v1);
  uint64_t from[VPT];
  bool live[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int e = v0 + u * kPackBlock + (int)threadIdx.x;
    live[u] = e < v1;
    from[u] = live[u] ? reinterpret_cast<uint64_t>(src) + (uint64_t)e * 16 : 0;
  }
  copy_chunk<VPT, false>(from, live, dst, v0, v1);
}

// Output row r is the row_bytes bytes at address rows_src[r] & ~15; bit 0 of
// an entry marks an embedding-table row, and a chunk holding one takes the
// pack's plain loads.
template <int VPT>
__global__ __launch_bounds__(kPackBlock) void k_gather(int32_t g0, int32_t g1, int32_t t1, int32_t t2, int32_t total,
                                                        uint64_t div_mul, int32_t div_shift, int32_t row_bytes,
                                                        const uint64_t* rows_src, uint8_t* dst) {
  extern __shared__ __align__(16) uint64_t s_src[];
  __shared__ int32_t s_table;
  int v0, v1;
  chunk_range<VPT>(g0, g1, t1, t2, total, &v0, &v1);
  auto div_row = [&](int e) { return (int)(((uint64_t)(uint32_t)e * div_mul) >> div_shift); };
  const int vpr = row_bytes >> 4;
  const int r0 = div_row(v0);
  const int rows = v1 > v0 ? div_row(v1 - 1) - r0 + 1 : 0;
  if (threadIdx.x == 0) s_table = 0;
  __syncthreads();
  for (int t = threadIdx.x; t < rows; t += kPackBlock) {
    const uint64_t x = rows_src[r0 + t];
    s_src[t] = x & ~(uint64_t)15;
    if (x & 1) s_table = 1;
  }
  __syncthreads();
  uint64_t from[VPT];
  bool live[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int e = v0 + u * kPackBlock + (int)threadIdx.x;
    live[u] = e < v1;
    from[u] = 0;
    if (live[u]) {
      const int row = div_row(e);
      from[u] = s_src[row - r0] + (uint64_t)(e - row * vpr) * 16;
    }
  }
  if (__builtin_amdgcn_readfirstlane(s_table)) copy_chunk<VPT, true>(from, live, dst, v0, v1);
  else copy_chunk<VPT, false>(from, live, dst, v0, v1);
}

// The pack's chunk geometry for `vecs` vectors of rows of row_bytes bytes.
static void plain_geometry(int64_t vecs, int64_t row_bytes, int n_cu, PackPlan* pl) {
  pl->vpt = vectors_per_thread(row_bytes);
  chunk_geometry(vecs, n_cu, pl);
}

hipError_t launch_copy(const void* src, void* dst, int64_t vecs, int64_t row_bytes, int n_cu, hipStream_t stream) {
  if (vecs <= 0) return hipSuccess;
  PackPlan pl{};
  plain_geometry(vecs, row_bytes, n_cu, &pl);
  const int grid = (int)(pl.g1 + (vecs - pl.t2 + kTail2Vecs - 1) / kTail2Vecs);
  if (pl.vpt == 2)
    hipLaunchKernelGGL(k_copy<2>, dim3(grid), dim3(kPackBlock), 0, stream, pl.g0, pl.g1, pl.t1, pl.t2, (int32_t)vecs,
                       (const uint8_t*)src, (uint8_t*)dst);
  else
    hipLaunchKernelGGL(k_copy<kVecsPerThread>, dim3(grid), dim3(kPackBlock), 0, stream, pl.g0, pl.g1, pl.t1, pl.t2,
                       (int32_t)vecs, (const uint8_t*)src, (uint8_t*)dst);
  return hipGetLastError();
}

hipError_t launch_gather(const uint64_t* rows_src, int32_t n_rows, int64_t row_bytes, void* dst, int n_cu,
                         hipStream_t stream) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t vecs = (int64_t)n_rows * (row_bytes >> 4);
  PackPlan pl{};
  plain_geometry(vecs, row_bytes, n_cu, &pl);
  const Divisors dv = make_divisors(row_bytes, 1, 16);
  const int grid = (int)(pl.g1 + (vecs - pl.t2 + kTail2Vecs - 1) / kTail2Vecs);
  const size_t lds = sizeof(uint64_t) * (size_t)std::min<int64_t>(n_rows, kChunkVecs / (row_bytes >> 4) + 2);
  if (pl.vpt == 2)
    hipLaunchKernelGGL(k_gather<2>, dim3(grid), dim3(kPackBlock), lds, stream, pl.g0, pl.g1, pl.t1, pl.t2,
                       (int32_t)vecs, dv.div_mul, dv.div_shift, (int32_t)row_bytes, rows_src, (uint8_t*)dst);
  else
    hipLaunchKernelGGL(k_gather<kVecsPerThread>, dim3(grid), dim3(kPackBlock), lds, stream, pl.g0, pl.g1, pl.t1,
                       pl.t2, (int32_t)vecs, dv.div_mul, dv.div_shift, (int32_t)row_bytes, rows_src, (uint8_t*)dst);
  return hipGetLastError();
}

hipError_t launch_write(const WriteArgs& a, hipStream_t stream) {
  const int64_t vecs = a.vis ? (int64_t)a.desc.n_vis * (a.row_bytes >> 4) : 0;
  const int grid = vecs > 0 ? (int)std::min<int64_t>((vecs + kChunkVecs - 1) / kChunkVecs, kWriteGrid) : 1;
  hipLaunchKernelGGL(k_write, dim3(grid), dim3(kPackBlock), sizeof(uint64_t) * (size_t)std::max(a.max_chunk_rows, 1),
                     stream, a);
  return hipGetLastError();
}

Divisors make_divisors(int64_t row_bytes, int64_t page_tokens, uint64_t page_bytes) {
  Divisors d{};
  // e / q for e < 2^31: with s = 31 + ceil(log2 q), m = ceil(2^s / q), e / q == (e * m) >> s.
  auto small = [](int64_t q, uint64_t* mul, int32_t* shift) {
    int c = 0;
    while ((1ll << c) < q) ++c;
    *shift = 31 + c;
    *mul = (uint64_t)(((1ull << *shift) + (uint64_t)q - 1) / (uint64_t)q);
  };
  small(row_bytes / 16, &d.div_mul, &d.div_shift);
  small(page_tokens, &d.pt_mul, &d.pt_shift);
  // GVA offset d < 2^52 by page_bytes: with c = ceil(log2 pb), N = max(52, 64 - c)
  // and s = N + c, m = ceil(2^s / pb) fits in 64 bits and d / pb == (d * m) >> s,
  // taken as the high 64 bits of the 128-bit product shifted by s - 64.
  int c = 0;
  while ((1ull << c) < page_bytes) ++c;
  const int sh = std::max(52, 64 - c) + c;
  d.pb_mul = (uint64_t)((((unsigned __int128)1 << sh) + page_bytes - 1) / page_bytes);
  d.pb_shift = sh - 64;
  return d;
}

hipError_t launch_cost(const SampleDesc* desc, const int32_t* slots, int32_t n, int64_t k,
                       int64_t* out_cost, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_cost, dim3((n + kBlock - 1) / kBlock), dim3(kBlock), 0, stream, desc,
                     slots, n, k, out_cost);
  return hipGetLastError();
}

}  // namespace fp
