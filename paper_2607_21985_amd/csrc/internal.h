// Internal declarations shared by the host-side C++ (host.cpp) and the HIP
// side (spdp.hip) of libspdp. Not part of the public ABI (include/spdp.h).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "spdp.h"

// One encoded matrix: the Tiled-CBC arrays on the host, their device copies,
// and the split-K workspace of the spMspV kernel.
struct spdp_matrix {
  int64_t rows = 0, cols = 0;
  int32_t tile_m = 0, tile_k = 0;
  int64_t n_stripes = 0, n_colblocks = 0, n_gtiles = 0;
  std::vector<uint32_t> tile_offset;
  std::vector<uint32_t> col_info;
  std::vector<uint64_t> bitmap;
  std::vector<uint16_t> values;  // fp16 bits (value_bits == 16)
  // value_bits 2..8: round-to-nearest codes, one byte each, in place of
  // `values`, and one fp32 scale per row
  int32_t value_bits = 16;
  std::vector<int8_t> codes;
  std::vector<float> scales;

  int device = -1;  // -1: host-only handle
  void* d_tile_offset = nullptr;
  void* d_col_info = nullptr;
  void* d_bitmap = nullptr;
  void* d_values = nullptr;  // fp16 values or codes
  void* d_scales = nullptr;

  // Split-K workspace: {fp32 partial sum, phase} pairs
  // [segments][batch][n_stripes*tile_m], and each row stripe's phase
  // (advanced on the device by every call).
  unsigned long long* d_partials = nullptr;
  size_t partial_floats = 0;  // capacity in pairs
  uint32_t* d_phase = nullptr;
  // Split-K partial sums of the prefill product (fp32, grown on demand).
  void* d_spmm_part = nullptr;
  size_t spmm_part_bytes = 0;
  // Workspaces replaced by a larger one: a HIP graph captured earlier still
  // names them, so they live until the handle is freed.
  std::vector<void*> retired;
};

namespace spdp {

// Records the detail text for the calling thread and returns `status`.
int fail(int status, const std::string& detail);
void clear_error();

// Validates shape/tile arguments and fills the host arrays of `m`.
int encode_host_arrays(const uint16_t* W, int64_t rows, int64_t cols,
                       int32_t tile_m, int32_t tile_k, spdp_matrix* m);
// The same with the weights quantized to `bits`-bit round-to-nearest codes
// (one fp32 scale per row) and stored one byte per code.
int encode_host_arrays_rtn(const uint16_t* W, int64_t rows, int64_t cols,
                           int32_t tile_m, int32_t tile_k, int32_t bits, spdp_matrix* m);

}  // namespace spdp
