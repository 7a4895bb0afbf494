// Device building blocks of the streaming kernels (forward and backward):
// address-space views for direct-to-LDS loads, the time-major LDS tile of the
// forward, the 16x16 MFMA operand paths, complex steps across a lane pair, and
// explicit memory-counter waits.
#pragma once

#include "common.h"

namespace res {

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// Time-major LDS tile of elements of ES bytes: rows of 128 bytes (the tile's
// channels), groups of 8 rows padded so that every group starts on a 16-byte
// boundary for the direct-to-LDS loads and row stores (bf16: +8 bytes, so the
// 8-byte operand gathers of 16 lanes from 16 different groups spread over the
// banks; float: +16 bytes).
constexpr int XROW = 128;
template <int ES> struct XLay {
  static constexpr int GRP = 8 * XROW + (ES == 2 ? 8 : 16);
  static constexpr int BYTES = (TILE_T / 8) * GRP;
  __device__ static __forceinline__ int off(int t) { return (t >> 3) * GRP + (t & 7) * XROW; }
};

// Compiler-level ordering of LDS accesses inside one wave (the LDS executes a
// wave's accesses in program order).
__device__ __forceinline__ void wave_lds_order() { asm volatile("" ::: "memory"); }

// ---------------------------------------------------------------------------
// Forward operands: every product contracts one chunk (16 steps).
//   FPath<float>: four v_mfma_f32_16x16x4_f32, slot (kk, q) = index 4q + kk:
//     lane (i, q) holds A[i][4q..4q+3], lane (n, q) holds B[4q..4q+3][n].
//   FPath<bf16_t>: split-bf16 on v_mfma_f32_16x16x16_bf16.  A per-channel
//     matrix A (from float64) is stored as Ah = bf16(A), Al = bf16(A - Ah); lane
//     (i, q) holds Ah[i][4q..4q+3] then Al[i][4q..4q+3] (16 bytes).  The
//     activations are exact in bf16; lane (n, q) holds x[16n+4q .. 16n+4q+3],
//     and two instructions give (Ah + Al) x (tables at ~2^-17 relative).
// In both, lane (n, q) of the activation operand reads tile rows 16n + 4q + r,
// r = 0..3: group 2n + (q >> 1), rows 4 (q & 1) + r.
// ---------------------------------------------------------------------------
template <typename TX> struct FPath;
template <> struct FPath<float> {
  typedef f4 AOp;
  typedef f4 XOp;
  __device__ static __forceinline__ AOp load_a(const void* p) { return load_f4(p); }
  __device__ static __forceinline__ AOp load_a_u4(uint4 u) {
    const f4 r = {__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w)};
    return r;
  }
  __device__ static __forceinline__ f4 mma(const AOp& a, const XOp& x, f4 c) { return mma_f32(a, x, c); }
  // (A x)^T: lane (i, q) gets columns 4q .. 4q+3 of row i of A x
  __device__ static __forceinline__ f4 mma_t(const XOp& x, const AOp& a, f4 c) { return mma_f32(x, a, c); }
  // y += U H for float32 states H (lane (n, q): components 4q .. 4q+3 of chunk n)
  typedef f4 UOp;
  __device__ static __forceinline__ UOp u_op(const f4& u) { return u; }
  __device__ static __forceinline__ f4 mma_u(const UOp& u, const f4& h, f4 c) { return mma_f32(u, h, c); }
  // the 4 consecutive channels ch0 .. ch0+3 (ch0 a multiple of 4), one 16-byte read per row
  __device__ static __forceinline__ void gather4(const char* xt, int ch0, int n, int q, XOp (&xv)[4]) {
    const char* p = xt + (2 * n + (q >> 1)) * XLay<4>::GRP + 4 * (q & 1) * XROW + ch0 * 4;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const f4 w = *reinterpret_cast<const f4*>(p + kk * XROW);
#pragma unroll
      for (int c = 0; c < 4; ++c) xv[c][kk] = w[c];
    }
  }
};
template <> struct FPath<bf16_t> {
  struct AOp {
    s4 hi, lo;
  };
  typedef s4 XOp;
  __device__ static __forceinline__ AOp load_a(const void* p) { return load_a_u4(*reinterpret_cast<const uint4*>(p)); }
  __device__ static __forceinline__ AOp load_a_u4(uint4 u) {
    AOp a;
    a.hi = __builtin_bit_cast(s4, make_uint2(u.x, u.y));
    a.lo = __builtin_bit_cast(s4, make_uint2(u.z, u.w));
    return a;
  }
  __device__ static __forceinline__ f4 mma(const AOp& a, const XOp& x, f4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.hi, x, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.lo, x, c, 0, 0, 0);
  }
  // (A x)^T: lane (i, q) gets columns 4q .. 4q+3 of row i of A x
  __device__ static __forceinline__ f4 mma_t(const XOp& x, const AOp& a, f4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x, a.hi, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x, a.lo, c, 0, 0, 0);
  }
  // y += U H for float32 states H (lane (n, q): components 4q .. 4q+3 of chunk n):
  // U (float32 table) and H split into bf16 halves, Uh Hh + Ul Hh + Uh Hl
  // (the omitted Ul Hl is ~2^-16 relative)
  typedef AOp UOp;
  __device__ static __forceinline__ UOp u_op(const f4& u) {
    UOp r;
    typedef __bf16 b4 __attribute__((ext_vector_type(4)));
    b4 hi, lo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      hi[i] = (__bf16)u[i];
      lo[i] = (__bf16)(u[i] - (float)hi[i]);
    }
    r.hi = __builtin_bit_cast(s4, hi);
    r.lo = __builtin_bit_cast(s4, lo);
    return r;
  }
  __device__ static __forceinline__ f4 mma_u(const UOp& u, const f4& h, f4 c) {
    // pairs rounded together; each remainder h - bf16(h) (exact: the two are
    // within a factor of two) as one bf16 dot product of the rounded pair with
    // (-1, 0) or (0, -1), accumulated onto h
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    // the two selectors live in registers: a packed bf16 operand given as a
    // 32-bit inline constant is not read as the pair written here
    uint32_t u10 = 0x0000BF80u, u01 = 0xBF800000u;
    asm volatile("" : "+v"(u10), "+v"(u01));
    const b2 m10 = __builtin_bit_cast(b2, u10), m01 = __builtin_bit_cast(b2, u01);
    uint32_t ph[2], pl[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const b2 hi = {(__bf16)h[2 * i], (__bf16)h[2 * i + 1]};
      ph[i] = __builtin_bit_cast(uint32_t, hi);
      const b2 lo = {(__bf16)__builtin_amdgcn_fdot2_f32_bf16(hi, m10, h[2 * i], false),
                     (__bf16)__builtin_amdgcn_fdot2_f32_bf16(hi, m01, h[2 * i + 1], false)};
      pl[i] = __builtin_bit_cast(uint32_t, lo);
    }
    const s4 bh = __builtin_bit_cast(s4, make_uint2(ph[0], ph[1]));
    const s4 bl = __builtin_bit_cast(s4, make_uint2(pl[0], pl[1]));
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(u.hi, bh, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(u.lo, bh, c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(u.hi, bl, c, 0, 0, 0);
  }
  // the 4 consecutive channels ch0 .. ch0+3 (ch0 a multiple of 4): element r of
  // channel c from row r (the compiler reads each row once and packs with byte
  // permutes)
  __device__ static __forceinline__ void gather4(const char* xt, int ch0, int n, int q, XOp (&xv)[4]) {
    const char* p = xt + (2 * n + (q >> 1)) * XLay<2>::GRP + 4 * (q & 1) * XROW + ch0 * 2;
    typedef unsigned short us4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      us4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = *reinterpret_cast<const unsigned short*>(p + r * XROW + c * 2);
      xv[c] = __builtin_bit_cast(s4, v);
    }
  }
};

__device__ __forceinline__ float swap_pair(float v) {  // value of the neighbouring lane (lane ^ 1)
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1,
                                                               0xF, 0xF, false));
}

// One complex multiply-add on the lane's component of a (re, im) lane pair:
// zr v + zs v' + add, with v' the value of lane i ^ 1 (the other component),
// zs = -Im z on the re lane and +Im z on the im lane.  The partner product is
// one fused multiply-add whose first operand is read across the pair (DPP
// quad_perm [1,0,3,2]).  A DPP read needs two wait states after a vector
// write of its source: the multiply-add on v, which must come between any
// write of v and this instruction, is one, the s_nop the other.
__device__ __forceinline__ float cfma_pair(float zr, float zs, float v, float add) {
  float acc = fmaf(zr, v, add);
  asm("s_nop 0\n\tv_fmac_f32_dpp %0, %1, %2 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf"
      : "+v"(acc)
      : "v"(v), "v"(zs));
  return acc;
}

// One 16-byte-per-lane load straight into LDS (64 lanes, 1 KB at lds) from
// base + off (base wave-uniform, off the lane's byte offset).  Issued as an
// opaque instruction: the compiler then does not wait for it before every later
// LDS read of the issuing wave (it cannot tell which buffer a read touches); the
// kernel waits for its own tiles explicitly (vmcnt) before the barrier that
// publishes them.
__device__ __forceinline__ void lds_dma16(const void* base, uint32_t off, const void* lds) {
  const uint32_t la = (uint32_t)(size_t)(lvoid_t*)lds;
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(la) : "memory");
}

// Wait until at most n (0 <= n <= 63) vector memory operations of the wave are
// outstanding (exp and lgkm counts not waited for).
__device__ __forceinline__ void wait_vmcnt(int n) {
  switch (n) {
#define RES_VMC(k) \
  case k: __builtin_amdgcn_s_waitcnt(0x0F70 | ((k) & 15) | (((k) >> 4) << 14)); break;
#define RES_VMC8(k) RES_VMC(k) RES_VMC(k + 1) RES_VMC(k + 2) RES_VMC(k + 3) RES_VMC(k + 4) RES_VMC(k + 5) \
  RES_VMC(k + 6) RES_VMC(k + 7)
    RES_VMC8(0) RES_VMC8(8) RES_VMC8(16) RES_VMC8(24) RES_VMC8(32) RES_VMC8(40) RES_VMC8(48) RES_VMC8(56)
#undef RES_VMC8
#undef RES_VMC
    default: __builtin_amdgcn_s_waitcnt(0x0F70); break;
  }
}

// 16-byte store of each lane to base + off (base wave-uniform), as an opaque
// instruction like lds_dma16, so that the compiler keeps the 64-bit base in
// scalar registers and the lane offset in one vector register.  A store of more
// than 8 bytes reads its data registers after issue: on gfx950 a vector write to
// them needs two wait states after the store, which the compiler's hazard
// tracking cannot see inside an asm statement, so the asm carries them.  The
// rows are outputs no work-group reads again, so the store is non-temporal
// (nt): it does not leave dirty lines in the L2 to be written back when the
// kernel ends (the forward at B4 L32K bf16: 65 to 60 us a launch).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st_row16(void* base, uint32_t off, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, %2 nt\n\ts_nop 1" ::"v"(off), "v"(v), "s"(base) : "memory");
}

// Transposition of the chunk sums of 4 channels across the wave: R[k] holds
// channel k with lane (i, q) carrying component i of chunks 4q .. 4q+3 (the
// transposed product layout); afterwards lane (i, c) holds component i of
// chunks 0 .. 15 of channel c in S[0 .. 15] (permlane swaps of 32 and 16 lanes).
__device__ __forceinline__ void lanes_to_chunks(const f4 (&R)[4], float (&S)[16]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint32_t v0 = __float_as_uint(R[0][r]), v1 = __float_as_uint(R[1][r]);
    const uint32_t v2 = __float_as_uint(R[2][r]), v3 = __float_as_uint(R[3][r]);
    const auto s02 = __builtin_amdgcn_permlane32_swap(v0, v2, false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(v1, v3, false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    S[r] = __uint_as_float(s01[0]);
    S[4 + r] = __uint_as_float(s01[1]);
    S[8 + r] = __uint_as_float(s23[0]);
    S[12 + r] = __uint_as_float(s23[1]);
  }
}

}  // namespace res
