// Coalesced movement of a [TILE_T x DW] activation tile between the [B][L][D]
// layout in HBM and a channel-major LDS tile [DW][TILE_T + pad].
//
// Global side: lane = channel, so one wave instruction touches one 128-byte row
// segment (bf16: 64 channels x 2 B; fp32: two rows of 32 channels x 4 B).
// LDS side: each lane packs 16 bytes of consecutive time steps of its channel,
// which is the layout the 16x16 MFMA operands read (4 consecutive steps of one
// channel per lane).
#pragma once

#include "common.h"

namespace res {

template <typename T, int DW>
struct TileGeom {
  static constexpr int R = 64 / DW;                    // rows per wave instruction
  static constexpr int NL = TILE_T / (R * NWAVES);     // rows per lane
  static constexpr int EPW = 16 / (int)sizeof(T);      // elements per 16-byte LDS access
  static constexpr int PITCH = TILE_T + EPW;           // LDS row pitch (elements), +16 B pad
};

// Load rows [t0, t0 + TILE_T) x channels [d0, d0 + DW) of batch b; zero outside
// [0, L) x [0, D).
template <typename T, int DW>
__device__ __forceinline__ void load_tile(const T* __restrict__ g, T* s, int64_t b, int64_t t0,
                                          int d0, int64_t L, int D, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
  const int d = d0 + ch;
  const bool dok = d < D;
  const int64_t base = (b * L + t0 + tb) * (int64_t)D + d;
#pragma unroll
  for (int i = 0; i < G::NL; i += G::EPW) {
    T v[G::EPW];
#pragma unroll
    for (int e = 0; e < G::EPW; ++e) {
      const int64_t t = t0 + tb + i + e;
      v[e] = (dok && t < L) ? g[base + (int64_t)(i + e) * D] : T(0);
    }
    *reinterpret_cast<uint4*>(&s[ch * G::PITCH + tb + i]) = *reinterpret_cast<const uint4*>(v);
  }
}

template <typename T, int DW>
__device__ __forceinline__ void store_tile(T* __restrict__ g, const T* s, int64_t b, int64_t t0,
                                           int d0, int64_t L, int D, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
  const int d = d0 + ch;
  const bool dok = d < D;
  const int64_t base = (b * L + t0 + tb) * (int64_t)D + d;
#pragma unroll
  for (int i = 0; i < G::NL; i += G::EPW) {
    T v[G::EPW];
    *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(&s[ch * G::PITCH + tb + i]);
#pragma unroll
    for (int e = 0; e < G::EPW; ++e) {
      const int64_t t = t0 + tb + i + e;
      if (dok && t < L) g[base + (int64_t)(i + e) * D] = v[e];
    }
  }
}

}  // namespace res
