// Wavefront-wide scans for gfx950 built on DPP.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace taccl {

// Cross-lane moves through DPP (a VALU operand modifier, so no trip
// through the LDS crossbar as with ds_bpermute): row_shr:n reads lane i - n
// of the same 16-lane row, row_bcast:15 / :31 read lane 15 / 31 into the
// next row(s) selected by the row mask, wave_shr:1 reads lane i - 1. Lanes
// without a source (and rows outside the mask) read 0, the identity of the
// unsigned add and max used here.
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, Ctrl, RowMask, 0xf, false);
}
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  const uint32_t lo = dpp<Ctrl, RowMask>((uint32_t)v), hi = dpp<Ctrl, RowMask>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
constexpr int kRowShr = 0x110, kBcast15 = 0x142, kBcast31 = 0x143, kWaveShr1 = 0x138;

// inclusive scans over the 64 lanes of a wavefront (Hillis-Steele inside
// each row, then the row broadcasts)
__device__ __forceinline__ uint32_t wave_scan_add(uint32_t v) {
  v += dpp<kRowShr + 1>(v);
  v += dpp<kRowShr + 2>(v);
  v += dpp<kRowShr + 4>(v);
  v += dpp<kRowShr + 8>(v);
  v += dpp<kBcast15, 0xa>(v);
  v += dpp<kBcast31, 0xc>(v);
  return v;
}
__device__ __forceinline__ uint64_t wave_scan_max64(uint64_t v) {
  v = max(v, dpp64<kRowShr + 1>(v));
  v = max(v, dpp64<kRowShr + 2>(v));
  v = max(v, dpp64<kRowShr + 4>(v));
  v = max(v, dpp64<kRowShr + 8>(v));
  v = max(v, dpp64<kBcast15, 0xa>(v));
  v = max(v, dpp64<kBcast31, 0xc>(v));
  return v;
}
// inclusive scans over lanes 0..15 only (the other rows hold garbage)
__device__ __forceinline__ uint32_t row_scan_add(uint32_t v) {
  v += dpp<kRowShr + 1>(v);
  v += dpp<kRowShr + 2>(v);
  v += dpp<kRowShr + 4>(v);
  v += dpp<kRowShr + 8>(v);
  return v;
}
__device__ __forceinline__ uint64_t row_scan_max64(uint64_t v) {
  v = max(v, dpp64<kRowShr + 1>(v));
  v = max(v, dpp64<kRowShr + 2>(v));
  v = max(v, dpp64<kRowShr + 4>(v));
  v = max(v, dpp64<kRowShr + 8>(v));
  return v;
}
__device__ __forceinline__ uint64_t readlane64(uint64_t v, uint32_t lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint32_t wave_scan_max(uint32_t v) {
  v = max(v, dpp<kRowShr + 1>(v));
  v = max(v, dpp<kRowShr + 2>(v));
  v = max(v, dpp<kRowShr + 4>(v));
  v = max(v, dpp<kRowShr + 8>(v));
  v = max(v, dpp<kBcast15, 0xa>(v));
  v = max(v, dpp<kBcast31, 0xc>(v));
  return v;
}
// maximum over the wavefront, the same in every lane
__device__ __forceinline__ uint32_t wave_reduce_max(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_max(v), 63);
}
__device__ __forceinline__ uint64_t wave_reduce_max64(uint64_t v) {
  return readlane64(wave_scan_max64(v), 63);
}

}  // namespace taccl
