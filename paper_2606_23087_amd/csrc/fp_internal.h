// Internal layout shared by the host pool code and the HIP kernels of
// libflowpool. Not part of the public ABI (see include/flowpool.h).
#pragma once

#include <hip/hip_runtime.h>
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
constexpr int kMaxTileRows = 64;     // rows per workgroup tile in k_write
constexpr int kPackBlock = 256;      // threads per k_pack workgroup
constexpr int kVecsPerThread = 3;    // 16-byte vectors each k_pack thread moves (12 KiB chunks)
constexpr int kChunkVecs = kPackBlock * kVecsPerThread;   // output vectors per k_pack workgroup
constexpr int kInlineSamples = 64;   // sample headers passed by value to k_pack
constexpr int kInlineImages = 128;   // image pairs passed by value to k_pack
constexpr int kImgGroup = 8;       // image pairs read per scalar load group in k_pack
constexpr int kLenGroup = 8;       // sample lengths read per scalar load group in k_pack
constexpr int kWaveRows = 16;      // rows per wave resolved with scalar loads in k_pack
static_assert(kInlineSamples % kLenGroup == 0, "length groups tile the inline headers");
constexpr int kMaxPackSamples = 1024;  // per microbatch (bounds k_pack's LDS use)
constexpr int kMaxPackImages = 1024;

// Per-sample header of a microbatch, taken from the pool's host mirror of
// the sample metadata (the variable-length parts stay in device memory).
struct alignas(16) PackSample {
  int32_t len;        // rows = text + visual
  int32_t n_img;
  int32_t img_base;   // index of the sample's first (position, rows) pair
  int32_t n_text;
  int64_t text_off;   // metadata-arena byte offset of the text ids
  int64_t page_off;   // metadata-arena byte offset of the page GVAs
};
static_assert(sizeof(PackSample) == 32, "PackSample layout");

// Everything one pack launch needs, passed by value. Kernel arguments are
// captured at launch, so microbatches of up to kInlineSamples samples and
// kInlineImages images need no staging copy; larger ones point at a staged
// device copy of the same arrays.
struct PackArgs {
  const uint8_t* meta;        // device metadata arena
  const uint64_t* pte;        // device page table, index = (gva - gva_start) / page_bytes
  uint64_t gva_start;
  uint64_t page_bytes;
  const uint8_t* table;       // embedding table (may be null when no text row is copied)
  uint8_t* out;               // packed rows
  int32_t* cu;                // cu_seqlens or null
  int32_t* pos;               // position ids or null
  const PackSample* samples_dev;   // staged headers, or null = samples[]
  const int2* imgs_dev;            // staged image pairs, or null = imgs[]
  int32_t n;                  // samples
  int32_t n_imgs;             // image pairs
  int32_t n_tokens;           // total rows
  int32_t row_bytes;
  int32_t page_tokens;
  int32_t tier_mask;
  int32_t max_chunk_rows;     // rows one chunk can touch
  uint64_t div_mul;           // e / (row_bytes/16) == (e * div_mul) >> div_shift for e < 2^31
  int32_t div_shift;
  int32_t pt_shift;           // v / page_tokens == (v * pt_mul) >> pt_shift for v < 2^31
  uint64_t pt_mul;
  uint64_t pb_mul;            // d / page_bytes == umulhi64(d, pb_mul) >> pb_shift for d < 2^52
  int32_t pb_shift;
  alignas(16) int32_t lens[kInlineSamples];   // sample lengths, zero past n
  PackSample samples[kInlineSamples];
  int2 imgs[kInlineImages + kImgGroup];       // zero past n_imgs, so a group may overrun
};

struct WriteArgs {
  SampleDesc desc;            // descriptor to publish into the table
  SampleDesc* desc_table;
  int32_t slot;
  const uint8_t* meta;
  const uint64_t* pte;
  uint64_t gva_start;
  uint64_t page_bytes;
  const uint8_t* vis;         // producer rows, or null
  int32_t row_bytes;
  int32_t page_tokens;
  int32_t tile_rows;
};

size_t pack_lds_bytes(const PackArgs& a);
hipError_t launch_pack(const PackArgs& a, hipStream_t stream);
hipError_t launch_write(const WriteArgs& a, hipStream_t stream);
hipError_t launch_cost(const SampleDesc* desc, const int32_t* slots, int32_t n, int64_t k,
                       int64_t* out_cost, hipStream_t stream);

}  // namespace fp
