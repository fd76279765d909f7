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
constexpr int kInlineSlots = 256;    // sample slots passed by value to k_pack
constexpr int kMaxTileRows = 64;     // rows resolved per workgroup tile
constexpr int kMaxPackSamples = 8192;   // keeps the LDS prefix-sum array at <= 32 KiB

// Everything one pack launch needs, passed by value (kernel arguments are
// captured at launch, so no host staging buffer is involved for n <= 256).
struct PackArgs {
  const SampleDesc* desc;     // device sample table
  const uint8_t* meta;        // device metadata arena
  const uint64_t* pte;        // device page table, index = (gva - gva_start) / page_bytes
  uint64_t gva_start;
  uint64_t page_bytes;
  const uint8_t* table;       // embedding table (may be null when no text rows)
  uint8_t* out;               // packed rows
  int32_t* cu;                // cu_seqlens or null
  int32_t* pos;               // position ids or null
  const int32_t* slots_dev;   // slot list in device memory, or null = slots_inline
  int32_t n;                  // samples
  int32_t n_tokens;           // total rows
  int32_t row_bytes;
  int32_t page_tokens;
  int32_t tier_mask;
  int32_t tile_rows;          // rows per workgroup tile (<= kMaxTileRows)
  int32_t slots_inline[kInlineSlots];
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

hipError_t launch_pack(const PackArgs& a, hipStream_t stream);
hipError_t launch_write(const WriteArgs& a, hipStream_t stream);
hipError_t launch_cost(const SampleDesc* desc, const int32_t* slots, int32_t n, int64_t k,
                       int64_t* out_cost, hipStream_t stream);

}  // namespace fp
