// Internal layout shared by the host pool code and the HIP kernels of
// libflowpool. Not part of the public ABI (see include/flowpool.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fp {

// Device sample descriptor, one per resident sample slot (48 bytes).
// The variable-length parts live in the metadata arena at byte offsets:
//   page_off: uint64 GVA per page, in visual-row order      [n_pages]
//   img_off : int32 pairs (placeholder position, rows)       [n_img]
//   text_off: int32 text token ids                            [n_text]
struct alignas(16) SampleDesc {
  int32_t len;      // n_text + n_vis
  int32_t n_text;
  int32_t n_img;
  int32_t n_vis;
  int64_t page_off;
  int64_t img_off;
  int64_t text_off;
  int32_t n_pages;
  int32_t pad;
};
static_assert(sizeof(SampleDesc) == 48, "descriptor layout");

// Page-table entry: device-visible address of the physical page, low bits
// used as flags (page addresses are at least 16-byte aligned).
constexpr uint64_t PTE_VALID = 1ull;
constexpr uint64_t PTE_HOST = 2ull;
constexpr uint64_t PTE_ADDR_MASK = ~0xFull;

constexpr int kBlock = 256;          // threads per workgroup for all kernels
constexpr int kPackBlock = 256;      // threads per k_pack workgroup
constexpr int kVecsPerThread = 3;    // 16-byte vectors each k_pack thread moves (12 KiB chunks)
constexpr int kChunkVecs = kPackBlock * kVecsPerThread;   // output vectors per k_pack workgroup
// Rows of at least this many bytes are packed in 8 KiB chunks (2 vectors per
// thread) instead: measured faster from H 5120 up, slower at H 3584 and 4096.
constexpr int kSmallChunkRowBytes = 10240;
// The last chunks of a pack are smaller, so the final workgroups finish
// sooner and the launch drains faster: one wave of resident workgroups (CUs x
// kPackPerCU) gets chunks of kTail1Vecs (the full size when rows take 8 KiB
// chunks), half a wave then kTail2Vecs.
constexpr int kPackPerCU = 8;        // k_pack workgroups resident per CU (occupancy 8)
constexpr int kTail1Vecs = 512;
constexpr int kTail2Vecs = 256;
constexpr int kInlineSamples = 32;   // sample lengths passed by value to k_pack
constexpr int kInlineRuns = 160;     // runs passed by value to k_pack
constexpr int kBuckets = 64;         // row buckets of the run index
constexpr int kWaveRows = 16;        // rows per wave resolved with scalar loads in k_pack
constexpr int kMaxPackSamples = 1024;  // per microbatch (bounds the staged run table)
constexpr int kMaxPackImages = 1024;

// A run is a maximal stretch of packed rows of one sample that come from one
// place: text rows (ids read from the sample's text list) or image rows (the
// images between two text rows, which are consecutive in the sample's page
// list). The host lists a microbatch's runs in row order, so resolving a row
// is finding its run and one or two indexed loads. Metadata-arena offsets are
// kept as word indexes, so the arena is limited to kMaxMetaBytes.
struct alignas(16) PackRun {
  int32_t end;        // one past the run's last row
  int32_t head;       // first row of the run's sample; bit 31 set for a text run
  int32_t vdelta;     // image run: visual index of row r is r + vdelta
  int32_t word;       // text run: the id of row r is 32-bit word word + r of the
                      // arena; image run: the sample's page GVAs start at
                      // 64-bit word `word`, or, when its pages have
                      // consecutive GVAs, -1 - (page number of its first page)
};
static_assert(sizeof(PackRun) == 16, "PackRun layout");
constexpr int32_t kTextRun = INT32_MIN;
// A bit of PackArgs::tier_mask beside the two tier bits: chunks holding
// embedding-table rows read with plain loads, which let the device's 256 MB
// memory-side cache keep table rows between reads. Set for tables of at most
// kPlainTableMaxBytes: over uniform random rows, plain loads gather 9 % faster
// than non-temporal ones from a 1.09 GB table, break even near 3 GB, and
// are 1.5 % slower from a 4.3 GB one.
constexpr int32_t kTablePlainLoads = 4;
constexpr int64_t kPlainTableMaxBytes = 5ll << 29;   // 2.5 GiB
constexpr int64_t kMaxMetaBytes = 1ll << 33;

// What the pack kernel reads, passed by value. The run table (sample
// lengths, runs, bucket index) follows the scalar fields; kernel arguments
// are captured at launch, so a microbatch of up to kInlineSamples samples and
// kInlineRuns runs needs no staging copy. A larger one is copied to device
// memory first, laid out at the given byte offsets. For each row bucket b,
// brun[b] is a copy of the run holding row b << bucket_shift and bucket[b]
// that run's index, so a row of the same run is resolved with one load, and a
// later row steps on from there. The table capacities are template
// parameters: PackArgs is the general form, PackArgsSmall a compact one for
// microbatches of a few samples, whose smaller kernel arguments take less
// host time to launch.
template <int kSamples, int kRuns, int kBucketCount>
struct PackArgsT {
  const uint8_t* meta;        // device metadata arena
  const uint64_t* pte;        // device page table, index = (gva - gva_start) / page_bytes
  uint64_t gva_start;
  const uint8_t* table;       // embedding table (may be null when no text row is copied)
  uint8_t* out;               // packed rows
  int32_t* cu;                // cu_seqlens or null
  int32_t* pos;               // position ids or null
  int32_t off_runs;           // byte offsets from the table's start: the runs,
  int32_t off_brun;           // the bucket runs and the bucket index
  int32_t off_bucket;
  int32_t bucket_shift;       // buckets hold 2^bucket_shift rows
  int32_t n;                  // samples
  int32_t n_tokens;           // total rows
  int32_t row_bytes;
  int32_t page_tokens;
  int32_t tier_mask;          // FP_TIER_MASK_* bits, plus kTablePlainLoads
  uint64_t pt_mul;            // v / page_tokens == (v * pt_mul) >> pt_shift for v < 2^31
  uint64_t pb_mul;            // d / page_bytes == umulhi64(d, pb_mul) >> pb_shift for d < 2^52
  int32_t pt_shift;
  int32_t pb_shift;
  alignas(16) int32_t lens[kSamples];   // sample lengths (rows), in pack order
  alignas(16) PackRun runs[kRuns];
  alignas(16) PackRun brun[kBucketCount];
  uint16_t bucket[kBucketCount];
  static constexpr int kMaxSamples = kSamples, kMaxRuns = kRuns, kMaxBuckets = kBucketCount;
};
using PackArgs = PackArgsT<kInlineSamples, kInlineRuns, kBuckets>;
using PackArgsSmall = PackArgsT<8, 24, 16>;
// The pack's kernel arguments, 64 bytes of leading scalars (preloaded into
// registers) and this struct, stay within 4 KiB.
static_assert(sizeof(PackArgs) + 64 <= 4096, "kernel arguments stay within 4 KiB");
static_assert(offsetof(PackArgs, lens) == offsetof(PackArgsSmall, lens), "same scalar fields");

// A pack launch: the kernel's arguments and, host side, its geometry.
struct PackPlan {
  PackArgs a;
  const uint8_t* staged;      // staged run table, or null = the arrays in `a`
  bool small;                 // launch with PackArgsSmall (its table copied from `a`)
  int32_t n_runs, n_buckets;  // entries of the table in `a`
  int32_t max_chunk_rows;     // rows one chunk can touch
  int32_t g0, g1;             // workgroups [0, g0): full chunks; [g0, g1): kTail1Vecs; then kTail2Vecs
  int32_t t1, t2;             // first vectors of the two tail stages (t1 = g0 * full chunk)
  int32_t vpt;                // vectors per thread of a full chunk (2 or kVecsPerThread)
  uint64_t div_mul;           // e / (row_bytes/16) == (e * div_mul) >> div_shift for e < 2^31
  int32_t div_shift;
};

// Division constants of a pool (host-computed once): for e < 2^31,
// e / (row_bytes / 16) == (e * div_mul) >> div_shift and
// e / page_tokens == (e * pt_mul) >> pt_shift; for d < 2^52,
// d / page_bytes == umulhi64(d, pb_mul) >> pb_shift.
struct Divisors {
  uint64_t div_mul, pt_mul, pb_mul;
  int32_t div_shift, pt_shift, pb_shift;
};

// Workgroups of one producer write at most; a larger write loops over its
// chunks. (Smaller caps, 128 to 512, made writes slower and did not make the
// packs beside them measurably faster.)
constexpr int kWriteGrid = 1 << 16;

// The producer's write of one sample: its visual rows (contiguous at `vis`)
// are copied into its pages in chunks of kChunkVecs vectors, like a pack
// with source and destination exchanged.
struct WriteArgs {
  SampleDesc desc;            // descriptor to publish into the table
  SampleDesc* desc_table;
  int32_t slot;
  int32_t row_bytes;
  const uint8_t* meta;
  const uint64_t* pte;
  uint64_t gva_start;
  const uint8_t* vis;         // producer rows, or null
  int32_t page_tokens;
  int32_t max_chunk_rows;     // rows one chunk can touch
  Divisors dv;
};

size_t pack_lds_bytes(const PackPlan& pl);
Divisors make_divisors(int64_t row_bytes, int64_t page_tokens, uint64_t page_bytes);
// Chunk geometry of a pack (g0, g1, t1, t2) for a device with n_cu compute units.
void pack_chunks(PackPlan* pl, int n_cu);
hipError_t launch_pack(const PackPlan& pl, hipStream_t stream);
hipError_t launch_write(const WriteArgs& a, hipStream_t stream);
// Measurement aids with the pack's geometry: a plain copy of `vecs` 16-byte
// vectors (chunks sized as for rows of row_bytes), and a gather of n_rows
// rows of row_bytes from the device addresses rows_src[] into consecutive
// rows of dst.
hipError_t launch_copy(const void* src, void* dst, int64_t vecs, int64_t row_bytes, int n_cu, hipStream_t stream);
hipError_t launch_gather(const uint64_t* rows_src, int32_t n_rows, int64_t row_bytes, void* dst, int n_cu,
                         hipStream_t stream);
hipError_t launch_cost(const SampleDesc* desc, const int32_t* slots, int32_t n, int64_t k,
                       int64_t* out_cost, hipStream_t stream);

}  // namespace fp
