// Definitions shared by the two per-row kernels (one workgroup per row with
// the row streamed through LDS, and one workgroup per compute unit holding
// whole rows in registers).
#pragma once

#include <type_traits>

#include "device_common.h"
#include "filter_tile.h"

namespace profk {

// Radix digit of the refinement and fallback: 16-bit keys take two 8-bit
// passes (a 256-word histogram), 32-bit keys three 11-bit ones.
template <int DT> constexpr int row_digit() { return Elem<DT>::KEYBITS == 16 ? 8 : 11; }

// Buffer keys are stored at their own width (bf16 keys in 16 bits).
template <int DT> using RowKey = typename std::conditional<Elem<DT>::KEYBITS == 16, uint16_t, uint32_t>::type;

// Log-scale buckets a row key distance can fall in: 16-bit keys keep every
// distance below 2^16, so bf16 rows need only the first 1280.
template <int DT> constexpr uint32_t row_log_bins() { return Elem<DT>::KEYBITS == 16 ? 1280u : kLogBins; }

}  // namespace profk
