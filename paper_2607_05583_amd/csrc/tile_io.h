// Coalesced movement of a [TILE_T x DW] activation tile between the [B][L][D]
// layout in HBM and a channel-major LDS tile [DW][TILE_T + pad].
//
// Global side: lane = channel, so one wave instruction touches one 128-byte row
// segment (bf16: 64 channels x 2 B; fp32: two rows of 32 channels x 4 B).
// LDS side: each lane packs 16 bytes of consecutive time steps of its channel,
// which is the layout the MFMA operands read (consecutive steps of one channel
// per lane).  Full tiles take an unguarded path whose row address is
// wave-uniform (scalar base + per-lane channel offset); edge tiles guard every
// element and read zeros outside [0, L) x [0, D).
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

// Rows [t0, t0 + TILE_T) x channels [d0, d0 + DW) of batch b.
template <typename T, int DW, bool FULL>
__device__ __forceinline__ void load_tile(const T* __restrict__ g, T* s, int64_t b, int64_t t0,
                                          int d0, int64_t L, int D, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
  if (FULL) {
    // wave-uniform row base; per-lane offset = channel + row block
    const T* base = g + ((b * L + t0 + wave * G::NL) * (int64_t)D + d0);
    const uint32_t loff = (uint32_t)(ro * (TILE_T / G::R) * D + ch);
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) v[e] = base[(size_t)(i + e) * D + loff];
      *reinterpret_cast<uint4*>(&s[ch * G::PITCH + tb + i]) = *reinterpret_cast<const uint4*>(v);
    }
  } else {
    const int d = d0 + ch;
    const bool dok = d < D;
    const int64_t gbase = (b * L + t0 + tb) * (int64_t)D + d;
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) {
        const int64_t t = t0 + tb + i + e;
        v[e] = (dok && t < L) ? g[gbase + (int64_t)(i + e) * D] : T(0);
      }
      *reinterpret_cast<uint4*>(&s[ch * G::PITCH + tb + i]) = *reinterpret_cast<const uint4*>(v);
    }
  }
}

template <typename T, int DW, bool FULL>
__device__ __forceinline__ void store_tile(T* __restrict__ g, const T* s, int64_t b, int64_t t0,
                                           int d0, int64_t L, int D, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
  if (FULL) {
    T* base = g + ((b * L + t0 + wave * G::NL) * (int64_t)D + d0);
    const uint32_t loff = (uint32_t)(ro * (TILE_T / G::R) * D + ch);
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
      *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(&s[ch * G::PITCH + tb + i]);
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) base[(size_t)(i + e) * D + loff] = v[e];
    }
  } else {
    const int d = d0 + ch;
    const bool dok = d < D;
    const int64_t gbase = (b * L + t0 + tb) * (int64_t)D + d;
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
      *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(&s[ch * G::PITCH + tb + i]);
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) {
        const int64_t t = t0 + tb + i + e;
        if (dok && t < L) g[gbase + (int64_t)(i + e) * D] = v[e];
      }
    }
  }
}

// Runtime dispatch between the two paths.
template <typename T, int DW>
__device__ __forceinline__ void load_tile_any(const T* g, T* s, int64_t b, int64_t t0, int d0,
                                              int64_t L, int D, int tid) {
  if (t0 + TILE_T <= L && d0 + DW <= D)
    load_tile<T, DW, true>(g, s, b, t0, d0, L, D, tid);
  else
    load_tile<T, DW, false>(g, s, b, t0, d0, L, D, tid);
}
template <typename T, int DW>
__device__ __forceinline__ void store_tile_any(T* g, const T* s, int64_t b, int64_t t0, int d0,
                                               int64_t L, int D, int tid) {
  if (t0 + TILE_T <= L && d0 + DW <= D)
    store_tile<T, DW, true>(g, s, b, t0, d0, L, D, tid);
  else
    store_tile<T, DW, false>(g, s, b, t0, d0, L, D, tid);
}

// ---------------------------------------------------------------------------
// Register staging of a tile (prefetch of the next tile while the current one
// is being computed): lane (ch, ro) of each wave holds its NL rows of one
// channel, packed 16 bytes per EPW consecutive rows, exactly as they are laid
// out in the LDS tile.  32 VGPRs per lane for both element types.
// ---------------------------------------------------------------------------
template <typename T, int DW>
struct TileRegs {
  static constexpr int N = TileGeom<T, DW>::NL / TileGeom<T, DW>::EPW;
  uint4 v[N];
};

template <typename T, int DW, bool FULL>
__device__ __forceinline__ void tile_to_regs(const T* __restrict__ g, TileRegs<T, DW>& r, int64_t b,
                                             int64_t t0, int d0, int64_t L, int D, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
  if (FULL) {
    const T* base = g + ((b * L + t0 + wave * G::NL) * (int64_t)D + d0);
    const uint32_t loff = (uint32_t)(ro * (TILE_T / G::R) * D + ch);
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) v[e] = base[(size_t)(i + e) * D + loff];
      r.v[i / G::EPW] = *reinterpret_cast<const uint4*>(v);
    }
  } else {
    const int d = d0 + ch;
    const bool dok = d < D;
    const int64_t gbase = (b * L + t0 + tb) * (int64_t)D + d;
#pragma unroll
    for (int i = 0; i < G::NL; i += G::EPW) {
      T v[G::EPW];
#pragma unroll
      for (int e = 0; e < G::EPW; ++e) {
        const int64_t t = t0 + tb + i + e;
        v[e] = (dok && t < L) ? g[gbase + (int64_t)(i + e) * D] : T(0);
      }
      r.v[i / G::EPW] = *reinterpret_cast<const uint4*>(v);
    }
  }
}

template <typename T, int DW>
__device__ __forceinline__ void tile_to_regs_any(const T* g, TileRegs<T, DW>& r, int64_t b,
                                                 int64_t t0, int d0, int64_t L, int D, int tid) {
  if (t0 + TILE_T <= L && d0 + DW <= D)
    tile_to_regs<T, DW, true>(g, r, b, t0, d0, L, D, tid);
  else
    tile_to_regs<T, DW, false>(g, r, b, t0, d0, L, D, tid);
}

template <typename T, int DW>
__device__ __forceinline__ void regs_to_lds(const TileRegs<T, DW>& r, T* s, int tid) {
  typedef TileGeom<T, DW> G;
  const int lane = tid & 63, wave = tid >> 6;
  const int ch = lane % DW, ro = lane / DW;
  const int tb = ro * (TILE_T / G::R) + wave * G::NL;
#pragma unroll
  for (int i = 0; i < G::NL; i += G::EPW)
    *reinterpret_cast<uint4*>(&s[ch * G::PITCH + tb + i]) = r.v[i / G::EPW];
}

}  // namespace res
