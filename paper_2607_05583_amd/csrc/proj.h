// Shared pieces of the grouped projection on MFMA (proj.hip) and of the mixer
// epilogue fused with the output projection (epilogue.hip): operand types, the
// staging of a block-diagonal weight (or of its transpose, for the data
// gradient) into LDS in the operand layout, and the stores of one group's
// outputs.  Layouts as described in proj.hip.
#pragma once

#include "common.h"
#include "stream.h"

namespace res {

constexpr int GP_THREADS = 256;  // four waves
constexpr int GP_MAXOB = 8;      // output blocks of 16 per group: d_out/G <= 128
constexpr int GP_MAXP = 16;      // 16-byte pieces per lane and token tile: d_in * size <= 1024 bytes
constexpr int GP_FRAG = 64 * 16; // bytes of one weight fragment (16 per lane)
constexpr int GP_MAXLDS = 64 << 10;
// Work-groups per compute unit in the projection grids (measured at B4 L32K
// bf16): one weight streams best with 8 (26 us against 32 us with 2: work-groups
// that start while others compute keep loads in flight); two weights and the
// fused epilogue, at twice to four times the registers per lane, with 2.
constexpr int GP_WG_PER_CU_ONE = 8;
constexpr int GP_WG_PER_CU_TWO = 2;
constexpr int EP_WG_PER_CU = 2;
// Weight gradient: tokens per chunk (the contraction of one MFMA), waves and
// threads per work-group, output blocks per wave, 8 x 8 staging blocks per
// thread, work-groups at most (twice as many for a single gradient) and tokens
// per work-group at least (partials: 1 KB per output block and work-group).
constexpr int WT_T = 32;
constexpr int WT_WAVES = 8;
constexpr int WT_THREADS = 64 * WT_WAVES;
constexpr int WT_MAXB = 8;
constexpr int WT_MAXU = 1;
constexpr int WT_GRID = 256;
constexpr int WT_MIN_TOKENS = 128;

template <typename T>
struct GPGeo {
  static constexpr bool BF = sizeof(T) == 2;
  static constexpr int KC = BF ? 32 : 16;  // inputs per fragment
  static constexpr int VE = 16 / (int)sizeof(T);
};

__device__ __forceinline__ f4 gp_mma(const u32x4& a, const u32x4& b, f4 c, bf16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a), __builtin_bit_cast(bf8, b), c, 0, 0,
                                                 0);
}
__device__ __forceinline__ f4 gp_mma(const u32x4& a, const u32x4& b, f4 c, float) {
  return mma_f32(__builtin_bit_cast(f4, a), __builtin_bit_cast(f4, b), c);
}

__device__ __forceinline__ uint32_t gp_pack(float a, float b) {
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  const b2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// The weight W [G][di][dq] into LDS at dst as G * (di / KC) * (dq / 16)
// fragments of 1 KB: element (g, k, o) to fragment (g, k / KC, block of o), lane
// (i, q) and slot r.  Each of the nt threads (index tid) moves 16-byte runs of
// weight rows.
template <typename T>
__device__ __forceinline__ void gp_stage(char* dst_bytes, const T* __restrict__ W, int G, int di, int dq, int tid,
                                         int nt) {
  typedef GPGeo<T> GG;
  const int KB = di / GG::KC, OB = dq / 16;
  T* dst = reinterpret_cast<T*>(dst_bytes);
  const int nrun = G * di * (dq / GG::VE);
  for (int e = tid; e < nrun; e += nt) {
    const int o0 = (e % (dq / GG::VE)) * GG::VE, row = e / (dq / GG::VE);  // row = g di + k
    const int g = row / di, k = row % di;
    const u32x4 v = *reinterpret_cast<const u32x4*>(W + (size_t)row * dq + o0);
    const T* vs = reinterpret_cast<const T*>(&v);
    const int kb = k / GG::KC, kk = k % GG::KC;
    const int q = GG::BF ? kk >> 3 : (kk >> 2) & 3, r = GG::BF ? kk & 7 : kk & 3;
#pragma unroll
    for (int c = 0; c < GG::VE; ++c) {
      const int o = o0 + c, pb = o >> 5, oo = o & 31;
      int ob, i;
      if ((OB & 1) && 2 * pb == OB - 1) {
        ob = 2 * pb;
        i = oo;
      } else {
        ob = 2 * pb + ((oo >> 2) & 1);
        i = 4 * (oo >> 3) + (oo & 3);
      }
      const int f = (g * KB + kb) * OB + ob;
      dst[((size_t)f * 64 + i + 16 * q) * GG::VE + r] = vs[c];
    }
  }
}

// The transpose of W [G][di][dq] (contraction over dq, outputs over di, as the
// data gradient dy W^T takes it) into LDS at dst as G * (dq / KC) * (di / 16)
// fragments: element W[g][o][c] to fragment (g, c / KC, block of o), lane
// (i(o), q) and slot r with c % KC = VE q + r.  A 16-byte run of a weight row
// holds VE adjacent contraction indices of one output, which is one lane's
// slots, so every run is one 16-byte LDS store.
template <typename T>
__device__ __forceinline__ void gp_stage_t(char* dst_bytes, const T* __restrict__ W, int G, int di, int dq, int tid,
                                           int nt) {
  typedef GPGeo<T> GG;
  const int KB = dq / GG::KC, OB = di / 16, rpr = dq / GG::VE;
  const int nrun = G * di * rpr;
  for (int e = tid; e < nrun; e += nt) {
    const int c0 = (e % rpr) * GG::VE, row = e / rpr;  // row = g di + o
    const int g = row / di, o = row % di;
    const u32x4 v = *reinterpret_cast<const u32x4*>(W + (size_t)row * dq + c0);
    const int kb = c0 / GG::KC, q = (c0 % GG::KC) / GG::VE;
    const int pb = o >> 5, oo = o & 31;
    int ob, i;
    if ((OB & 1) && 2 * pb == OB - 1) {
      ob = 2 * pb;
      i = oo;
    } else {
      ob = 2 * pb + ((oo >> 2) & 1);
      i = 4 * (oo >> 3) + (oo & 3);
    }
    const int f = (g * KB + kb) * OB + ob;
    *reinterpret_cast<u32x4*>(dst_bytes + ((size_t)f * 64 + i + 16 * q) * 16) = v;
  }
}

// One group's OB output blocks (accumulators a[0 .. OB-1], MFMA D layout) of one
// token into its output row yr (the group's first output), lane q.
// With ACC the outputs' present values are added (in float32) before the
// rounding.
template <typename T, int MOB, bool ACC = false>
__device__ __forceinline__ void gp_store(T* yr, const f4 (&a)[MOB], int OB, int q) {
#pragma unroll
  for (int ob = 0; ob < MOB; ob += 2) {
    if (ob >= OB) continue;
    f4 a0 = a[ob];
    if (ob + 1 < OB) {  // a pair: 8 adjacent outputs from 32 (ob / 2) + 8 q
      f4 a1 = a[ob + 1];
      T* yp = yr + 16 * ob + 8 * q;
      if constexpr (ACC) {
        if constexpr (GPGeo<T>::BF) {
          const u32x4 o = *reinterpret_cast<const u32x4*>(yp);
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            a0[2 * r] += __uint_as_float(o[r] << 16);
            a0[2 * r + 1] += __uint_as_float(o[r] & 0xffff0000u);
            a1[2 * r] += __uint_as_float(o[2 + r] << 16);
            a1[2 * r + 1] += __uint_as_float(o[2 + r] & 0xffff0000u);
          }
        } else {
          a0 += *reinterpret_cast<const f4*>(yp);
          a1 += *reinterpret_cast<const f4*>(yp + 4);
        }
      }
      if constexpr (GPGeo<T>::BF) {
        *reinterpret_cast<u32x4*>(yp) =
            u32x4{gp_pack(a0[0], a0[1]), gp_pack(a0[2], a0[3]), gp_pack(a1[0], a1[1]), gp_pack(a1[2], a1[3])};
      } else {
        *reinterpret_cast<f4*>(yp) = a0;
        *reinterpret_cast<f4*>(yp + 4) = a1;
      }
    } else {  // the unpaired last block: 4 adjacent outputs from 16 ob + 4 q
      T* yp = yr + 16 * ob + 4 * q;
      if constexpr (ACC) {
        if constexpr (GPGeo<T>::BF) {
          const uint2 o = *reinterpret_cast<const uint2*>(yp);
          a0[0] += __uint_as_float(o.x << 16);
          a0[1] += __uint_as_float(o.x & 0xffff0000u);
          a0[2] += __uint_as_float(o.y << 16);
          a0[3] += __uint_as_float(o.y & 0xffff0000u);
        } else {
          a0 += *reinterpret_cast<const f4*>(yp);
        }
      }
      if constexpr (GPGeo<T>::BF)
        *reinterpret_cast<uint2*>(yp) = make_uint2(gp_pack(a0[0], a0[1]), gp_pack(a0[2], a0[3]));
      else
        *reinterpret_cast<f4*>(yp) = a0;
    }
  }
}

}  // namespace res
