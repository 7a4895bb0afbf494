// Device-side building blocks shared by the gfx950 kernels of the resonant mixing
// library: tile geometry, element conversion, 16x16 MFMA wrappers, workspace
// layout and the kernel argument blocks.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace res {

typedef short s4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;

// ---------------------------------------------------------------------------
// Tile geometry.  A tile is one batch row b, TILE_T consecutive time steps and
// D_W consecutive channels.  Inside a tile the time axis is cut into NCHUNK
// chunks of CHUNK steps; per channel, the chunk-local causal convolution, the
// chunk end-states and the carry correction are 16x16 matrix products whose
// columns are the tile's chunks.
// ---------------------------------------------------------------------------
constexpr int CHUNK = 16;
constexpr int NCHUNK = 16;
constexpr int TILE_T = CHUNK * NCHUNK;  // 256
constexpr int NTHREADS = 256;           // 4 waves of 64
constexpr int NWAVES = NTHREADS / 64;
constexpr int MODES_PER_GROUP = 8;      // one 16-row MFMA block = 8 complex modes
constexpr int MG_MAX = 2;               // M <= 16
constexpr int RES_M_MAX_DEV = MODES_PER_GROUP * MG_MAX;

// Channels per tile: 128-byte rows of the [B][L][D] layout.
template <typename T> constexpr int tile_channels() { return 128 / (int)sizeof(T); }

// ---------------------------------------------------------------------------
// Element conversion
// ---------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) {
  // round to nearest even (gfx950 converts in hardware)
  return __builtin_bit_cast(bf16_t, (__bf16)v);
}

// ---------------------------------------------------------------------------
// 16x16 MFMA operands.  Lane = i + 16 q (i = 0..15, q = 0..3); results D[4q + r][n],
// r = 0..3, sit in lane (n, q) for every instruction used here.
//
// Products with an activation operand (x or dy) use Path<T> of the activation
// type T:
//   Path<float>: a 16-deep contraction as four v_mfma_f32_16x16x4_f32 whose
//     slot (kk, q) is index 4q + kk: lane (i, q) holds A[i][4q..4q+3] and lane
//     (n, q) holds B[4q..4q+3][n].
//   Path<bf16_t>: split-bf16 on v_mfma_f32_16x16x32_bf16.  A per-channel matrix
//     A (from float64) is stored as A = Ah + Al with Ah = bf16(A), Al =
//     bf16(A - Ah); lane (i, q) holds [Ah | Al][i][8q..8q+7] (Ah for q < 2, Al
//     for q >= 2).  The activation operand is duplicated along the 32-deep
//     contraction (lane (n, q) holds B[8(q&1)..8(q&1)+7][n]); activations are
//     exact in bf16, so one instruction gives (Ah + Al) B with the tables at
//     ~2^-17 relative precision.
// Products of two computed float32 quantities (carried states, cross sums) use
// mma_f32: the fp32 layout of Path<float>, whatever the activation type.
// ---------------------------------------------------------------------------
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f4 mma_f32(const f4& a, const f4& b, f4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], c, 0, 0, 0);
  return c;
}
__device__ __forceinline__ f4 load_f4(const void* p) { return *reinterpret_cast<const f4*>(p); }

template <typename TX> struct Path;

template <> struct Path<float> {
  typedef f4 AOp;  // table operand (16 bytes per lane)
  typedef f4 XOp;  // activation operand
  __device__ static __forceinline__ int x_off(int li, int lq) { return li * 16 + lq * 4; }
  __device__ static __forceinline__ XOp load_x(const float* p) { return *reinterpret_cast<const f4*>(p); }
  __device__ static __forceinline__ AOp load_a(const void* p) { return *reinterpret_cast<const f4*>(p); }
  __device__ static __forceinline__ f4 mma(const f4& a, const f4& b, f4 c) { return mma_f32(a, b, c); }
};

template <> struct Path<bf16_t> {
  typedef bf8 AOp;
  typedef bf8 XOp;
  __device__ static __forceinline__ int x_off(int li, int lq) { return li * 16 + (lq & 1) * 8; }
  __device__ static __forceinline__ XOp load_x(const bf16_t* p) { return *reinterpret_cast<const bf8*>(p); }
  __device__ static __forceinline__ AOp load_a(const void* p) { return *reinterpret_cast<const bf8*>(p); }
  __device__ static __forceinline__ f4 mma(const bf8& a, const bf8& b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

// ---------------------------------------------------------------------------
// Carried-state rows of the multi-group forward: the state entering chunk n of
// (channel, mode m) is put into the chunk's row of a scan buffer as float32
// (re, im) at floats 2m, 2m+1; the MFMA lanes read the row back as the B
// operand of y += U H (float32 layout, four v_mfma_f32_16x16x4_f32).
// ---------------------------------------------------------------------------
struct StateRow {
  __device__ static __forceinline__ void put(float* row, int m, float2 h) {
    *reinterpret_cast<float2*>(row + 2 * m) = h;
  }
  __device__ static __forceinline__ f4 apply(const f4& u, const float* row, int lq, f4 acc) {
    return mma_f32(u, *reinterpret_cast<const f4*>(row + 4 * lq), acc);
  }
};

// exact product of two activation gathers (K16 layout)
__device__ __forceinline__ f4 mma_k16_act(const s4& a, const s4& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mma_k16_act(const f4& a, const f4& b, f4 c) { return mma_f32(a, b, c); }

// ---------------------------------------------------------------------------
// Complex helpers (float2 / double2 as re, im)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cfma(float2 a, float2 b, float2 c) {  // a*b + c
  return make_float2(fmaf(a.x, b.x, fmaf(-a.y, b.y, c.x)), fmaf(a.x, b.y, fmaf(a.y, b.x, c.y)));
}
__device__ __forceinline__ double2 zmul(double2 a, double2 b) {
  return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 zfma(double2 a, double2 b, double2 c) {
  return make_double2(fma(a.x, b.x, fma(-a.y, b.y, c.x)), fma(a.x, b.y, fma(a.y, b.x, c.y)));
}

// ---------------------------------------------------------------------------
// Problem geometry and workspace layout (host and device)
// ---------------------------------------------------------------------------
struct Geometry {
  int64_t B, L, D, M;
  int DW;        // channels per tile
  int NB;        // channel blocks
  int Dp;        // padded channels NB * DW
  int MG;        // mode groups of 8
  int Mp;        // padded modes 8 * MG
  int64_t P;     // tiles along time
  int last_len;  // valid steps of the last tile (1..TILE_T)
};

__host__ __device__ inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Bytes of one 16x16 operand matrix in the parameter table: 64 lanes x 16 bytes
// (4 float32, or 8 bf16 = hi | lo halves) for both operand paths.
constexpr size_t TAB_LANE_BYTES = 16;
constexpr size_t TAB_MAT_BYTES = 64 * TAB_LANE_BYTES;

// Number of 16x16 operand matrices per channel in the parameter table.
// Forward: T, then per mode group V[g], U[g].  Backward: Tt, then per mode group
// Eq[g], Er[g], Ub[g].  Matrices that multiply an activation use the activation
// path's layout; those that multiply computed float32 states (the forward's U,
// the backward's Ub) use the float32 layout.
__host__ __device__ constexpr int fwd_mats(int MG) { return 1 + 2 * MG; }
__host__ __device__ inline bool fwd_mat_is_state(int mat) { return mat > 0 && (mat - 1) % 2 == 1; }
__host__ __device__ constexpr int bwd_mats(int MG) { return 1 + 3 * MG; }
__host__ __device__ inline bool bwd_mat_is_state(int mat) { return mat > 0 && (mat - 1) % 3 == 2; }

// Per-mode float scalars of the tables (fwd and bwd).
struct ModeScalars {
  float2 lam;     // lambda
  float2 mu;      // lambda^CHUNK
  float2 mu8;     // lambda^(TILE_T / 2): the hop over half a tile (8 chunks)
  float2 lamT;    // lambda^TILE_T
  float2 lamTail; // lambda^(jstar+1): the steps of the last chunk up to t = L-1
};
// Per-mode float64 scalars for the cross-tile carry chain.
struct ModeCarry {
  double2 lamT;    // lambda^TILE_T
  double2 lamEll;  // lambda^last_len
  double2 mu8;     // lambda^(TILE_T / 2)
  double2 lam1;    // lambda
  double2 c;       // c = amp e^{i phase}
  double2 ephi;    // e^{i phase}
};

// Offsets (bytes) of the workspace regions.
struct WsLayout {
  size_t tab, scal, carryc, agg, carry, alast, part, q0, total;
};

}  // namespace res
