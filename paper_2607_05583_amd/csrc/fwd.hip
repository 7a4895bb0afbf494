// Forward resonant mixing, prompt state and parameter tables for gfx950.
//
// Operator (Sec. 3.1 kernel, Sec. 3.2 causal convolution, Sec. 3.3 recurrence):
//   y[t] = sum_{s<=t} K[t-s] x[s] + Re sum_m c_m lambda_m^(t+1) h0_m,
//   K[tau] = Re sum_m c_m lambda_m^tau.
// Chunked form used here (chunk of CHUNK = 16 steps, chunk n starts at 16 n):
//   y_loc[16n+i] = sum_{k<=i} K[i-k] x[16n+k]                 T  (16x16 lower Toeplitz)
//   S_m[n]      = sum_k lambda_m^(15-k) x[16n+k]              V  (16 x 16: 8 modes, re/im)
//   H_m[n+1]    = lambda_m^16 H_m[n] + S_m[n]                  scan over chunks
//   y[16n+i]    = y_loc[16n+i] + Re sum_m c_m lambda_m^(i+1) H_m[n]   U (16 x 16)
// where H_m[n] is the state entering chunk n.  Per channel the three products
// are 16x16 MFMAs whose 16 columns are the chunks of one tile (256 steps); all
// chunks share the per-channel matrices because the filter is time invariant.
// The single-kernel forward (M <= 8) cuts each row into segments of tiles: a
// segment computes its own end state, combines the published end states of the
// segments before it into its entering state, and then runs the chunk scan and
// the output products tile by tile.  With more than 8 modes the same steps run
// as three kernels (tile aggregates, carry fold, output pass).
#include "common.h"
#include "kernels.h"
#include "tile_io.h"

namespace res {

// ---------------------------------------------------------------------------
// Parameter tables.  One block per (padded) channel.  Every power lambda^n used
// (n = 0..16, 128, 256, last_len, 16 j for j < 16 and seg_steps n for n <= 16)
// is evaluated directly as exp(-gamma n) (cos(omega n), sin(omega n)) in
// float64 from the products gamma n and omega n (float32 times an integer:
// exact below 2^29), and c = a (cos phi, sin phi); all are independent, so
// the block does them in one parallel round (the time of this kernel is its
// longest dependent chain, not its work).  Entries are rounded once to the
// operand type.
// ---------------------------------------------------------------------------
constexpr int PREP_THREADS = 512;

template <typename TA, bool BWD>
__global__ __launch_bounds__(PREP_THREADS) void prep_kernel(const float* __restrict__ gamma,
                                                   const float* __restrict__ omega,
                                                   const float* __restrict__ amp,
                                                   const float* __restrict__ phase, int D, int M,
                                                   int MG, int last_len, int seg_steps,
                                                   TA* __restrict__ tab,
                                                   ModeScalars* __restrict__ scal,
                                                   ModeCarry* __restrict__ cc,
                                                   float2* __restrict__ mpow,
                                                   float2* __restrict__ spow,
                                                   uint32_t* __restrict__ flags, int64_t nflags) {
  // lambda^0..16, then lambda^128, lambda^256, lambda^last_len
  constexpr int NPW = CHUNK + 1 + 3;
  const int d = blockIdx.x;
  const int Mp = MODES_PER_GROUP * MG;
  __shared__ double2 pw[MODES_PER_GROUP * MG_MAX][NPW];
  __shared__ double2 cm[MODES_PER_GROUP * MG_MAX];  // c
  __shared__ double taps[CHUNK + 1];

  if (flags != nullptr)  // single-kernel forward: header words, then unpublished payload words
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nflags;
         i += (int64_t)gridDim.x * blockDim.x)
      flags[i] = i < SEG_HEADER_WORDS ? 0u : PAY_EMPTY_WORD;
  const bool dvalid = d < D;
  // one round: the table powers and c, then lambda^(16 j) as [d][j][Mp] and
  // lambda^(seg_steps n) as [d][n][Mp], both straight to global memory
  const int n_pw = Mp * (NPW + 1), n_mp = mpow ? Mp * CHUNK : 0, n_sp = spow ? Mp * (CHUNK + 1) : 0;
  for (int t = threadIdx.x; t < n_pw + n_mp + n_sp; t += blockDim.x) {
    if (t >= n_pw) {
      const int u = t - n_pw;
      const bool is_mp = u < n_mp;
      const int v = is_mp ? u : u - n_mp;
      const int m = v % Mp, j = v / Mp;
      const double n = is_mp ? (double)(CHUNK * j) : (double)seg_steps * (double)j;
      double2 z = make_double2(0.0, 0.0);
      if (dvalid && m < M) {
        double sn, cs;
        sincos((double)omega[d * M + m] * n, &sn, &cs);
        const double e = exp(-(double)gamma[d * M + m] * n);
        z = make_double2(e * cs, e * sn);
      }
      if (is_mp)
        mpow[((size_t)d * CHUNK + j) * Mp + m] = make_float2((float)z.x, (float)z.y);
      else
        spow[((size_t)d * (CHUNK + 1) + j) * Mp + m] = make_float2((float)z.x, (float)z.y);
      continue;
    }
    const int m = t / (NPW + 1), k = t % (NPW + 1);
    const bool valid = dvalid && m < M;
    if (k < NPW) {
      const int n = k <= CHUNK          ? k
                    : k == CHUNK + 1 ? TILE_T / 2
                    : k == CHUNK + 2 ? TILE_T
                                     : last_len;
      double2 z = make_double2(0.0, 0.0);
      if (valid) {
        double sn, cs;
        sincos((double)omega[d * M + m] * n, &sn, &cs);
        const double e = exp(-(double)gamma[d * M + m] * n);
        z = make_double2(e * cs, e * sn);
      }
      pw[m][k] = z;
    } else {
      double2 z = make_double2(0.0, 0.0);
      if (valid) {
        double sn, cs;
        sincos((double)phase[d * M + m], &sn, &cs);
        const double av = (double)amp[d * M + m];
        z = make_double2(av * cs, av * sn);
      }
      cm[m] = z;
    }
  }
  __syncthreads();
  for (int m = threadIdx.x; m < Mp; m += blockDim.x) {
    const double2 lam = pw[m][1], lH = pw[m][CHUNK + 1], lT = pw[m][CHUNK + 2];
    ModeScalars ms;
    ms.lam = make_float2((float)lam.x, (float)lam.y);
    ms.mu = make_float2((float)pw[m][CHUNK].x, (float)pw[m][CHUNK].y);
    ms.mu8 = make_float2((float)lH.x, (float)lH.y);
    ms.lamT = make_float2((float)lT.x, (float)lT.y);
    const int ntail = last_len > 0 ? (last_len - 1) % CHUNK + 1 : 0;
    ms.lamTail = make_float2((float)pw[m][ntail].x, (float)pw[m][ntail].y);
    scal[(size_t)d * Mp + m] = ms;
    ModeCarry mc;
    mc.lamT = lT;
    mc.lamEll = pw[m][CHUNK + 3];
    mc.mu8 = lH;
    cc[(size_t)d * Mp + m] = mc;
  }
  for (int tau = threadIdx.x; tau <= CHUNK; tau += blockDim.x) {  // K[tau] = Re sum_m c lambda^tau
    double s = 0.0;
    for (int m = 0; m < Mp; ++m) s += cm[m].x * pw[m][tau].x - cm[m].y * pw[m][tau].y;
    taps[tau] = s;
  }
  __syncthreads();

  auto part = [](double2 z, int p) { return p ? z.y : z.x; };
  // entry (mat, i, k) of the per-channel 16x16 matrices, k = contraction index
  auto entry = [&](int mat, int i, int k) -> double {
    if (!BWD) {
      if (mat == 0) return (i >= k) ? taps[i - k] : 0.0;          // T[i][k] = K[i-k]
      const int g = (mat - 1) / 2;
      if ((mat - 1) % 2 == 0)                                     // V[comp i][k] = lambda^(15-k)
        return part(pw[g * 8 + i / 2][CHUNK - 1 - k], i & 1);
      const int m = g * 8 + k / 2;                                // U[i][comp k] = c lambda^(i+1)
      const double2 z = zmul(cm[m], pw[m][i + 1]);
      return (k & 1) ? -z.y : z.x;
    }
    if (mat == 0) return (k >= i) ? taps[k - i] : 0.0;            // Tt[j=i][k] = K[k-i]
    const int g = (mat - 1) / 5, s = (mat - 1) % 5;
    const int mi = g * 8 + i / 2;
    switch (s) {
      case 0: return part(pw[mi][k], i & 1);                      // Eq[comp i][k] = lambda^k
      case 1: return k * part(pw[mi][k], i & 1);                  // Er = k lambda^k
      case 2: return part(pw[mi][CHUNK - k], i & 1);              // Xs = lambda^(16-k)
      case 3: return (CHUNK - k) * part(pw[mi][CHUNK - k], i & 1);  // Xw = (16-k) lambda^(16-k)
      default: {                                                  // Ub[j=i][comp k] = c lambda^(16-i)
        const int m = g * 8 + k / 2;
        const double2 z = zmul(cm[m], pw[m][CHUNK - i]);
        return (k & 1) ? -z.y : z.x;
      }
    }
  };

  // Store in the per-lane operand layout: 16 bytes per lane.
  const int nm = BWD ? bwd_mats(MG) : fwd_mats(MG);
  for (int task = threadIdx.x; task < nm * 64; task += blockDim.x) {
    const int mat = task / 64, l = task % 64, i = l % 16, q = l / 16;
    const bool state_mat = BWD ? bwd_mat_is_state(mat) : fwd_mat_is_state(mat);
    uint4 out;
    if (sizeof(TA) == 4 || state_mat) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (float)entry(mat, i, 4 * q + r);
      out = *reinterpret_cast<const uint4*>(v);
    } else if (!BWD) {  // Ah[i][4q..4q+3], then Al[i][4q..4q+3]
      bf16_t v[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const double e = entry(mat, i, 4 * q + r);
        const bf16_t hi = from_f32<bf16_t>((float)e);
        v[r] = hi;
        v[4 + r] = from_f32<bf16_t>((float)(e - (double)to_f32(hi)));
      }
      out = *reinterpret_cast<const uint4*>(v);
    } else {  // [Ah | Al][i][8q..8q+7] (32-deep contraction, activation duplicated)
      bf16_t v[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const double e = entry(mat, i, 8 * (q & 1) + r);
        const bf16_t hi = from_f32<bf16_t>((float)e);
        v[r] = (q < 2) ? hi : from_f32<bf16_t>((float)(e - (double)to_f32(hi)));
      }
      out = *reinterpret_cast<const uint4*>(v);
    }
    static_assert(sizeof(uint4) == TAB_LANE_BYTES, "one table lane is 16 bytes");
    reinterpret_cast<uint4*>(tab)[((size_t)d * nm + mat) * 64 + l] = out;
  }
}

// ---------------------------------------------------------------------------
// Forward tile machinery.
//
// A tile is one batch row b, 256 steps and DW channels (64 bf16 / 32 fp32, so a
// time row of the tile is one 128-byte segment).  Four waves each own CPW = DW/4
// channels, handled in groups of 4.
//
// LDS.  The drive tile is time-major: 32 groups of 8 rows (128 B each) with a
// 4-byte pad per group, filled by direct-to-LDS 16-byte loads.  Each output
// channel overwrites its own drive column once its products are done, and the
// tile leaves as 16-byte row stores.  Each wave has a scan buffer
// [4 channels][16 chunks][16 MG floats]: chunk states go from the MFMA layout
// (lane (n, q) holds components 4q..4q+3 of chunk n) to the scan layout, and
// the carried states come back the same way.
//
// Scan layout: lane 16 c + 2 m + h holds channel c of the group, mode m, for the
// chunk half h (chunks 8h .. 8h+7).  With A_h the end state of half h from a
// zero start (A_h = sum_j mu^(7-j) S[8h+j], mu = lambda^16), the tile's own
// end state is mu^8 A_0 + A_1, and half 1 of a tile entered with state c enters
// with mu^8 c + A_0.
//
// Per-tile records ([tile][DW * Mp] float4, slot q = wave * 32 PAIRS + 32 (grp
// MG + g) + 8 c + m): the aggregate kernel writes (A_0, A_1); the carry kernel
// writes the entry states (c, mu^8 c + A_0) of both halves.
// ---------------------------------------------------------------------------
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

// Drive tile [t0, t0 + 256) x [d0, d0 + DW) of row b into the time-major LDS
// tile; zeros outside [0, L) x [0, D).  full: the whole tile is in range and the
// rows are 16-byte aligned (direct-to-LDS loads); the caller waits (vmcnt) and
// synchronises before reading.
template <typename TX>
__device__ __forceinline__ void tile_load(char* xt, const TX* x, int64_t b, int64_t t0, int d0,
                                          int64_t L, int D, bool full, int tid) {
  constexpr int DW = tile_channels<TX>(), XE = (int)sizeof(TX);
  const int lane = tid & 63, wave = tid >> 6;
  if (full) {
    const char* src = reinterpret_cast<const char*>(x) + ((b * L + t0) * D + d0) * XE;
    const int64_t rowb = (int64_t)D * XE;
#pragma unroll
    for (int i = 0; i < TILE_T / 8 / NWAVES; ++i) {
      const int g = wave * (TILE_T / 8 / NWAVES) + i;
      const char* s = src + (int64_t)(8 * g + (lane >> 3)) * rowb + (lane & 7) * 16;
      __builtin_amdgcn_global_load_lds((gvoid_t*)s, (lvoid_t*)(xt + g * XLay<XE>::GRP), 16, 0, 0);
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      TX v = from_f32<TX>(0.f);
      if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
      *reinterpret_cast<TX*>(xt + XLay<XE>::off(t) + c * XE) = v;
    }
  }
}

template <typename TY>
__device__ __forceinline__ void tile_store(TY* y, const char* xt, int64_t b, int64_t t0, int d0,
                                           int64_t L, int D, bool full, int tid) {
  constexpr int DW = tile_channels<TY>(), YE = (int)sizeof(TY);
  const int lane = tid & 63, wave = tid >> 6;
  if (full) {
    char* dst = reinterpret_cast<char*>(y) + ((b * L + t0) * D + d0) * YE;
    const int64_t rowb = (int64_t)D * YE;
#pragma unroll
    for (int i = 0; i < TILE_T / 8 / NWAVES; ++i) {
      const int g = wave * (TILE_T / 8 / NWAVES) + i;
      const uint4 v = *reinterpret_cast<const uint4*>(xt + g * XLay<YE>::GRP + lane * 16);
      *reinterpret_cast<uint4*>(dst + (int64_t)(8 * g + (lane >> 3)) * rowb + (lane & 7) * 16) = v;
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      if (t0 + t < L && d0 + c < D)
        y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + XLay<YE>::off(t) + c * YE);
    }
  }
}

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
  __device__ static __forceinline__ AOp load_a(const void* p) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
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
    // pairs rounded together; the float value of each rounded half read back
    // from the packed word (low half: shift, high half: mask)
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    uint32_t ph[2], pl[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const b2 hi = {(__bf16)h[2 * i], (__bf16)h[2 * i + 1]};
      ph[i] = __builtin_bit_cast(uint32_t, hi);
      const b2 lo = {(__bf16)(h[2 * i] - __uint_as_float(ph[i] << 16)),
                     (__bf16)(h[2 * i + 1] - __uint_as_float(ph[i] & 0xFFFF0000u))};
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

// Outputs of the 4 consecutive channels ch0 .. ch0+3 of a group (MFMA D layout,
// lane (n, q) holds rows 16n + 4q + r) into the time-major LDS tile.
template <typename TY>
__device__ __forceinline__ void put_y4(char* xt, int ch0, int n, int q, const f4 (&acc)[4]) {
  // rows 16n + 4q + r: group 2n + (q >> 1), rows 4 (q & 1) + r
  char* dst = xt + (2 * n + (q >> 1)) * XLay<sizeof(TY)>::GRP + 4 * (q & 1) * XROW + ch0 * (int)sizeof(TY);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (sizeof(TY) == 2) {
      typedef __bf16 bf4 __attribute__((ext_vector_type(4)));
      const bf4 v = {(__bf16)acc[0][r], (__bf16)acc[1][r], (__bf16)acc[2][r], (__bf16)acc[3][r]};
      *reinterpret_cast<bf4*>(dst + r * XROW) = v;
    } else {
      const f4 v = {acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
      *reinterpret_cast<f4*>(dst + r * XROW) = v;
    }
  }
}

__device__ __forceinline__ float swap_pair(float v) {  // value of the neighbouring lane (lane ^ 1)
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1,
                                                               0xF, 0xF, false));
}

// float32 outputs straight from the MFMA registers: rows t .. t+3 of the 4
// channels d .. d+3, 16 bytes per row where all 4 channels exist.
__device__ __forceinline__ void put_y4_global(float* y, const f4 (&acc)[4], int64_t b, int64_t t, int d,
                                              int64_t L, int D) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (t + r >= L) break;
    float* dst = y + (b * L + t + r) * (int64_t)D + d;
    if (d + 4 <= D && (D & 3) == 0) {
      const f4 v = {acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
      *reinterpret_cast<f4*>(dst) = v;
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (d + c < D) dst[c] = acc[c][r];
    }
  }
}

template <typename TX, int MG>
struct FwdTile {
  typedef FPath<TX> PT;
  static constexpr int DW = tile_channels<TX>();
  static constexpr int CPW = DW / NWAVES;     // channels per wave
  static constexpr int NGRP = CPW / 4;       // scan groups of 4 channels
  static constexpr int NSTR = 16 * MG;       // floats per chunk row of the scan buffer
  static constexpr int CSTR = 16 * NSTR + 8; // floats per channel of the scan buffer
  static constexpr int WBUF = 4 * CSTR;      // floats per wave
  static constexpr int NM = fwd_mats(MG);
  static constexpr int PAIRS = NGRP * MG;    // (group, mode group) states per scan lane
};

// S = V x for the 4 channels of a group into the wave's scan buffer.
template <typename TX, int MG>
__device__ __forceinline__ void group_states(const char* xt, float* wb, int ch0,
                                             const typename FPath<TX>::AOp (&vop)[4][MG],
                                             typename FPath<TX>::XOp (&xv)[4], int ln, int lq) {
  typedef FwdTile<TX, MG> F;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  FPath<TX>::gather4(xt, ch0, ln, lq, xv);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int g = 0; g < MG; ++g)
      *reinterpret_cast<f4*>(&wb[k * F::CSTR + ln * F::NSTR + g * 16 + lq * 4]) =
          FPath<TX>::mma(vop[k][g], xv[k], zero);
  }
}

// ---------------------------------------------------------------------------
// Aggregate kernel: per tile and scan lane, the half-tile end states (A_0, A_1)
// from a zero start; the last tile of a row also gives the state at t = L-1
// from a zero start at its first step (alast).
// ---------------------------------------------------------------------------
template <typename TX, int MG>
__global__ __launch_bounds__(NTHREADS, MG == 1 ? 4 : 2) void fwd_agg_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  constexpr int DW = F::DW, CPW = F::CPW, NGRP = F::NGRP, XE = (int)sizeof(TX);
  __shared__ __align__(16) char xt[XLay<XE>::BYTES];
  __shared__ __align__(16) float sbuf[NWAVES * F::WBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 15, lq = lane >> 4;
  const int sh = lane & 1, sm = (lane >> 1) & 7, sc = lane >> 4;
  const int nchains = (int)(a.B * a.NB);
  const int64_t tile = blockIdx.x;
  const int64_t p = tile / nchains;
  const int chain = (int)(tile % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t t0 = p * TILE_T;
  const bool last = (p == a.P - 1);
  const bool full = a.fast_io && t0 + TILE_T <= a.L && d0 + DW <= a.D;
  const int cw0 = wave * CPW;
  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* wb = sbuf + wave * F::WBUF;

  typename PT::AOp vop[4][MG];
  auto fetch_v = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int g = 0; g < MG; ++g)
        vop[k][g] = PT::load_a(tab + (size_t)(d0 + cw0 + 4 * grp + k) * F::NM * TAB_MAT_BYTES +
                               lane * TAB_LANE_BYTES + (1 + 2 * g) * TAB_MAT_BYTES);
  };
  fetch_v(0);
  tile_load<TX>(xt, reinterpret_cast<const TX*>(a.x), b, t0, d0, a.L, a.D, full, tid);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  float4* rec = reinterpret_cast<float4*>(a.agg) + (size_t)tile * DW * a.Mp + wave * 32 * F::PAIRS;
#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp) {
    typename PT::XOp xv[4];
    group_states<TX, MG>(xt, wb, cw0 + 4 * grp, vop, xv, ln, lq);
    if (grp + 1 < NGRP) fetch_v(grp + 1);
    wave_lds_order();
    const int ch = cw0 + 4 * grp + sc;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const int m = g * 8 + sm;
      const float2 mu = a.scal[(size_t)(d0 + ch) * a.Mp + m].mu;
      float2 run = make_float2(0.f, 0.f), hl = run;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (8 * sh + j == nstar) hl = run;  // state entering chunk nstar (from this half's start)
        const float2 sv =
            *reinterpret_cast<const float2*>(&wb[sc * F::CSTR + (8 * sh + j) * F::NSTR + g * 16 + 2 * sm]);
        run = cfma(mu, run, sv);
      }
      const float2 oth = make_float2(swap_pair(run.x), swap_pair(run.y));
      const float2 A0 = sh ? oth : run, A1 = sh ? run : oth;
      if (sh == 0) rec[(grp * MG + g) * 32 + sc * 8 + sm] = make_float4(A0.x, A0.y, A1.x, A1.y);
      if (last && a.alast != nullptr && sh == (nstar >> 3)) {
        // state at t = L-1 from a zero start at the tile's first step
        const ModeScalars ms = a.scal[(size_t)(d0 + ch) * a.Mp + m];
        if (sh == 1) {  // half 0 contributes mu^(nstar - 8) A_0
          float2 w = A0;
          for (int i = 8; i < nstar; ++i) w = cmul(ms.mu, w);
          hl = make_float2(hl.x + w.x, hl.y + w.y);
        }
        for (int i = 0; i <= jstar; ++i) {
          const TX xv1 = *reinterpret_cast<const TX*>(xt + XLay<XE>::off(nstar * CHUNK + i) + ch * XE);
          hl = cfma(ms.lam, hl, make_float2(to_f32(xv1), 0.f));
        }
        a.alast[((size_t)b * a.Dp + d0 + ch) * a.Mp + m] = hl;
      }
    }
    wave_lds_order();
  }
}

// ---------------------------------------------------------------------------
// Carry kernel: for every (row, channel, mode) the states entering each tile.
// The tiles of a row are cut into at most 64 segments of 16 * 2^k tiles;
// thread (pair, segment) folds its segment's aggregates from zero (float64), the
// segment entry states follow from the segment aggregates in order, and each
// thread replays its segment to write the entry states of both tile halves
// (c, mu^8 c + A_0).  The last
// segment also writes the state at t = L-1: lambda^last_len c_last + alast.
// The fold order is fixed by P alone, so the result is bitwise reproducible.
// ---------------------------------------------------------------------------
constexpr int CARRY_SEG_MAX = 64;  // segments per row (threads per pair)
constexpr int CARRY_BLOCK = 16;    // records loaded together

__global__ __launch_bounds__(256) void fwd_carry_kernel(FwdArgs a, int seg_len, int nseg, int nsegp,
                                                        int pairs_per_tile, int cpw, int pairs_w) {
  __shared__ double2 sg[256];  // segment aggregates, then entry states
  const int tid = threadIdx.x;
  const int pw = 256 / nsegp;                    // pairs per block
  const int seg = tid / pw, pl = tid % pw;
  const int64_t pair = (int64_t)blockIdx.x * pw + pl;  // (chain, q)
  const int nchains = (int)(a.B * a.NB);
  const bool valid = pair < (int64_t)nchains * pairs_per_tile && seg < nseg;
  const int chain = (int)(pair / pairs_per_tile), q = (int)(pair % pairs_per_tile);
  // slot q -> (channel, mode): q = wave * 32 PAIRS + 32 (grp MG + g) + 8 c + m
  const int MG = a.Mp / 8;
  const int wv = q / (32 * pairs_w), s = q % (32 * pairs_w);
  const int grp = s / (32 * MG), g = (s / 32) % MG, c = (s / 8) % 4, m8 = s % 8;
  const int ch = wv * cpw + 4 * grp + c, m = g * 8 + m8;
  const int64_t b = chain / a.NB;
  const int d = (chain % a.NB) * (cpw * NWAVES) + ch;
  const float4* agg = reinterpret_cast<const float4*>(a.agg);
  float4* car = reinterpret_cast<float4*>(a.car);

  double2 lamT = make_double2(0.0, 0.0), mu8 = lamT;
  if (valid) {
    const ModeCarry cc = a.cc[(size_t)d * a.Mp + m];
    lamT = cc.lamT;
    mu8 = cc.mu8;
  }
  const int64_t p0 = (int64_t)seg * seg_len;
  const int nsub = seg_len / CARRY_BLOCK;
  // records of tile p0 + i of this (row, pair): base[i * stride]
  const size_t stride = (size_t)nchains * pairs_per_tile;
  const float4* base = agg + (size_t)(p0 * nchains + chain) * pairs_per_tile + q;
  float4* cbase = car + (size_t)(p0 * nchains + chain) * pairs_per_tile + q;
  const int64_t nloc = valid ? (a.P - p0 < seg_len ? a.P - p0 : seg_len) : 0;  // tiles of this segment
  float4 rec[CARRY_BLOCK];
  // pass 1: the segment's end state from zero over its tiles before the row's last
  double2 acc = make_double2(0.0, 0.0);
  for (int sb = 0; sb < nsub; ++sb) {
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i) {
      const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
      rec[i] = li < nloc ? base[li * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i)
      if (p0 + (int64_t)sb * CARRY_BLOCK + i < a.P - 1)
        acc = zfma(lamT, acc, zfma(mu8, make_double2(rec[i].x, rec[i].y), make_double2(rec[i].z, rec[i].w)));
  }
  sg[tid] = acc;
  __syncthreads();
  // entry state of this segment: h0, then hop over the earlier segments in order
  double2 lamS = lamT;  // lambda^(256 seg_len), seg_len a power of two
  for (int e = seg_len; e > 1; e >>= 1) lamS = zmul(lamS, lamS);
  double2 ent = make_double2(0.0, 0.0);
  if (valid && a.h0 != nullptr && d < a.D && m < a.M) {
    const float* h = a.h0 + ((size_t)(b * a.D + d) * a.M + m) * 2;
    ent = make_double2(h[0], h[1]);
  }
  for (int s2 = 0; s2 < seg; ++s2) ent = zfma(lamS, ent, sg[s2 * pw + pl]);
  if (!valid) return;
  // pass 2: replay, writing the entry states of every tile of the segment
  double2 cst = ent;
  for (int sb = 0; sb < nsub; ++sb) {
    if (nsub > 1) {  // a single block is still in registers
#pragma unroll
      for (int i = 0; i < CARRY_BLOCK; ++i) {
        const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
        rec[i] = li < nloc ? base[li * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i) {
      const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
      if (li < nloc) {
        const double2 A0 = make_double2(rec[i].x, rec[i].y), A1 = make_double2(rec[i].z, rec[i].w);
        const double2 half = zfma(mu8, cst, A0);
        if (car != nullptr)
          cbase[li * stride] = make_float4((float)cst.x, (float)cst.y, (float)half.x, (float)half.y);
        if (p0 + li == a.P - 1) {
          if (a.h_out != nullptr && d < a.D && m < a.M) {
            const double2 lE = a.cc[(size_t)d * a.Mp + m].lamEll;
            const float2 al = a.alast[((size_t)b * a.Dp + d) * a.Mp + m];
            const double2 hL = zfma(lE, cst, make_double2(al.x, al.y));
            float* ho = a.h_out + ((size_t)(b * a.D + d) * a.M + m) * 2;
            ho[0] = (float)hL.x;
            ho[1] = (float)hL.y;
          }
        } else {
          cst = zfma(lamT, cst, zfma(mu8, A0, A1));
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Apply kernel: each scan lane runs its 8 chunks from its half's entry state
// and leaves the state entering every chunk in the scan buffer; then per channel
// y = T x + U H on MFMA, written over the drive column; the tile leaves as rows.
// ---------------------------------------------------------------------------
template <typename TX, typename TY, int MG>
__global__ __launch_bounds__(NTHREADS, MG == 1 ? 4 : 2) void fwd_apply_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  constexpr int DW = F::DW, CPW = F::CPW, NGRP = F::NGRP;
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) char xt[XLay<sizeof(TX)>::BYTES];
  __shared__ __align__(16) float sbuf[NWAVES * F::WBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 15, lq = lane >> 4;
  const int sh = lane & 1, sm = (lane >> 1) & 7, sc = lane >> 4;
  const int nchains = (int)(a.B * a.NB);
  const int64_t tile = blockIdx.x;
  const int64_t p = tile / nchains;
  const int chain = (int)(tile % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t t0 = p * TILE_T;
  const bool full = a.fast_io && t0 + TILE_T <= a.L && d0 + DW <= a.D;
  const int cw0 = wave * CPW;
  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* wb = sbuf + wave * F::WBUF;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};

  auto tab_of = [&](int ch) {
    return tab + (size_t)(d0 + ch) * F::NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
  };
  typedef StateRow SO;
  typename PT::AOp vop[4][MG], top[4];
  f4 uop[4][MG];
  auto fetch_v = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int g = 0; g < MG; ++g) vop[k][g] = PT::load_a(tab_of(cw0 + 4 * grp + k) + (1 + 2 * g) * TAB_MAT_BYTES);
  };
  auto fetch_tu = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const char* tp = tab_of(cw0 + 4 * grp + k);
      top[k] = PT::load_a(tp);
#pragma unroll
      for (int g = 0; g < MG; ++g) uop[k][g] = load_f4(tp + (2 + 2 * g) * TAB_MAT_BYTES);
    }
  };
  // entry state of this lane's half, per (group, mode group)
  const float2* car = reinterpret_cast<const float2*>(reinterpret_cast<const float4*>(a.car) +
                                                      (size_t)tile * DW * a.Mp + wave * 32 * F::PAIRS);
  float2 ent[NGRP][MG];
#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp)
#pragma unroll
    for (int g = 0; g < MG; ++g) ent[grp][g] = car[2 * ((grp * MG + g) * 32 + sc * 8 + sm) + sh];
  fetch_v(0);
  fetch_tu(0);
  tile_load<TX>(xt, reinterpret_cast<const TX*>(a.x), b, t0, d0, a.L, a.D, full, tid);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp) {
    typename PT::XOp xv[4];
    group_states<TX, MG>(xt, wb, cw0 + 4 * grp, vop, xv, ln, lq);
    if (grp + 1 < NGRP) fetch_v(grp + 1);
    wave_lds_order();
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const float2 mu = a.scal[(size_t)(d0 + cw0 + 4 * grp + sc) * a.Mp + g * 8 + sm].mu;
      float2 run = ent[grp][g];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float* row = &wb[sc * F::CSTR + (8 * sh + j) * F::NSTR + g * 16];
        const float2 sv = *reinterpret_cast<const float2*>(row + 2 * sm);
        SO::put(row, sm, run);  // state entering chunk 8 sh + j
        run = cfma(mu, run, sv);
      }
    }
    wave_lds_order();
    f4 acc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[k] = PT::mma(top[k], xv[k], zero);
#pragma unroll
      for (int g = 0; g < MG; ++g)
        acc[k] = SO::apply(uop[k][g], &wb[k * F::CSTR + ln * F::NSTR + g * 16], lq, acc[k]);
    }
    if (SEPY)
      put_y4_global(reinterpret_cast<float*>(a.y), acc, b, t0 + ln * CHUNK + lq * 4, d0 + cw0 + 4 * grp,
                    a.L, a.D);
    else
      put_y4<TY>(xt, cw0 + 4 * grp, ln, lq, acc);
    if (grp + 1 < NGRP) fetch_tu(grp + 1);
    wave_lds_order();
  }
  if (!SEPY) {
    __syncthreads();
    tile_store<TY>(reinterpret_cast<TY*>(a.y), xt, b, t0, d0, a.L, a.D, full, tid);
  }
}

// ---------------------------------------------------------------------------
// Single-kernel forward over row segments (one mode group, M <= 8).
//
// A work-group (8 waves) owns seg_len consecutive tiles of one chain (batch row
// b, channel block); each wave owns CW channels of the tile and keeps their
// operands in registers for the whole segment.  Per channel the state MFMA
// S = V x leaves, in lane (n, q), the drives of chunk n for the modes 2q and
// 2q+1; everything on the chunk axis then runs across the 16 lanes of a row.
//   pass 1  per tile, lane-wise acc = lambda^256 acc + mu^(15-n) S; the row sum
//           of acc is the segment's own end state from a zero start (agg_s);
//   carry   per wave (its channels form their own sub-chain): publish agg_s,
//           wait for the aggregates of all earlier segments of the row and
//           fold them, with the row's initial state, into the state entering
//           the segment (a fixed-order weighted sum, lanes in parallel);
//   pass 2  the segment streams again: per tile and channel, the entering state
//           c is added to lane 0 as mu c, the chunk recurrence
//           Q[n] = mu Q[n-1] + S[n] is a four-step prefix scan over the row
//           (shifts 1, 2, 4, 8 with multipliers mu, mu^2, mu^4, mu^8), the
//           state entering chunk n is Q[n-1] (c for n = 0) and feeds
//           y = T x + U H directly as the float32 MFMA operand; Q[15] is the
//           next tile's entering state.
// Tiles stream through three LDS tile buffers; wave 0 alone issues the
// direct-to-LDS loads (two tiles in flight), the other waves store the output
// rows.  Work-groups take segments in ticket order (time-major over the chains),
// so every wait is on a smaller ticket, which a running work-group took and
// publishes without waiting; every wait is bounded.  Payloads and flags are agent-coherent (device-scope)
// accesses; a publisher completes its payload stores before the flag store.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st_agent(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
// the two modes of a lane as (re, im, re, im)
__device__ __forceinline__ void st_agent4(float2* p, f4 v) {
  st_agent(p, make_float2(v[0], v[1]));
  st_agent(p + 1, make_float2(v[2], v[3]));
}
__device__ __forceinline__ f4 ld_agent4(const float2* p) {
  const float2 u = ld_agent(p), w = ld_agent(p + 1);
  const f4 r = {u.x, u.y, w.x, w.y};
  return r;
}
__device__ __forceinline__ uint32_t ld_flag(const uint32_t* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(uint32_t* f, uint32_t v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Upper bound on window polls (about a second); reached only if a predecessor
// never publishes, which the ticket order rules out.  The wave then starts from
// the row's initial state and records the event in the error word.
constexpr uint32_t SPIN_LIMIT = 1u << 20;
constexpr uint32_t PAY_EMPTY = PAY_EMPTY_WORD;

// Complex arithmetic on the two modes of a lane, (re_a, im_a, re_b, im_b).
__device__ __forceinline__ f4 c2mul(const f4& a, const f4& b) {
  f4 r;
  r[0] = fmaf(a[0], b[0], -a[1] * b[1]);
  r[1] = fmaf(a[0], b[1], a[1] * b[0]);
  r[2] = fmaf(a[2], b[2], -a[3] * b[3]);
  r[3] = fmaf(a[2], b[3], a[3] * b[2]);
  return r;
}
__device__ __forceinline__ f4 c2fma(const f4& a, const f4& b, const f4& c) {  // a b + c
  f4 r;
  r[0] = fmaf(a[0], b[0], fmaf(-a[1], b[1], c[0]));
  r[1] = fmaf(a[0], b[1], fmaf(a[1], b[0], c[1]));
  r[2] = fmaf(a[2], b[2], fmaf(-a[3], b[3], c[2]));
  r[3] = fmaf(a[2], b[3], fmaf(a[3], b[2], c[3]));
  return r;
}
__device__ __forceinline__ f4 mode_pair(float2 u, float2 w) {
  const f4 r = {u.x, u.y, w.x, w.y};
  return r;
}

// Lane moves inside rows of 16 lanes (DPP).  BOUND0: lanes without a source
// lane read zero; otherwise they keep `old`.
constexpr int DPP_ROW_SHL(int n) { return 0x100 + n; }   // lane i <- lane i + n
constexpr int DPP_ROW_SHR(int n) { return 0x110 + n; }   // lane i <- lane i - n
constexpr int DPP_QUAD(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }
constexpr int DPP_ROW_MIRROR = 0x140;                    // lane i <- lane 15 - i
constexpr int DPP_ROW_HALF_MIRROR = 0x141;               // lane i <- lane 7 - i (per half row)
template <int CTRL, bool BOUND0>
__device__ __forceinline__ f4 dpp4(const f4& old, const f4& v) {
  f4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float o = old[i], x = v[i];  // scalars: a vector element is no lvalue for bit_cast
    r[i] = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, o),
                                                                 __builtin_bit_cast(int, x), CTRL,
                                                                 0xF, 0xF, BOUND0));
  }
  return r;
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

// Sum over the 16 lanes of each row, in every lane of the row (the same order in
// every lane, so the copies agree bitwise).
__device__ __forceinline__ f4 row_sum(f4 v) {
  v += dpp4<DPP_QUAD(1, 0, 3, 2), false>(v, v);
  v += dpp4<DPP_QUAD(2, 3, 0, 1), false>(v, v);
  v += dpp4<DPP_ROW_HALF_MIRROR, false>(v, v);
  v += dpp4<DPP_ROW_MIRROR, false>(v, v);
  return v;
}

template <typename TX>
struct SegGeo {
  static constexpr int DW = tile_channels<TX>();
  static constexpr int NW = sizeof(TX) == 2 ? 16 : 8;  // waves
  static constexpr int CW = DW / NW;    // channels per wave (4)
  // 16 waves: one channel at a time through the scan (one LDS slot per wave);
  // 8 waves: four channels at a time (four slots per wave)
  static constexpr int SLOTS = NW == 16 ? 1 : 4;
  static constexpr int NG = CW / 4;     // operand gathers of 4 channels per wave
  static constexpr int NT = 64 * NW;    // threads
  // tile buffers; the waves w with w % NBUF == u load the tiles of buffer u
  static constexpr int NBUF = seg_bufs((int)sizeof(TX));
  static_assert(NBUF <= NW, "a loading wave per buffer");
};

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

// Wait until at most n vector memory operations of the wave are outstanding
// (n <= 15; exp and lgkm counts not waited for).
__device__ __forceinline__ void wait_vmcnt(int n) {
  switch (n) {
#define RES_VMCNT(k) \
  case k: __builtin_amdgcn_s_waitcnt(0x0F70 | k); break;
    RES_VMCNT(0) RES_VMCNT(1) RES_VMCNT(2) RES_VMCNT(3) RES_VMCNT(4) RES_VMCNT(5) RES_VMCNT(6) RES_VMCNT(7)
    RES_VMCNT(8) RES_VMCNT(9) RES_VMCNT(10) RES_VMCNT(11) RES_VMCNT(12) RES_VMCNT(13) RES_VMCNT(14)
#undef RES_VMCNT
    default: __builtin_amdgcn_s_waitcnt(0x0F70 | 15); break;
  }
}

// 16-byte store of each lane to base + off (base wave-uniform), as an opaque
// instruction like lds_dma16, so that the compiler keeps the 64-bit base in
// scalar registers and the lane offset in one vector register.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st_row16(void* base, uint32_t off, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, %2" ::"v"(off), "v"(v), "s"(base) : "memory");
}

// Direct-to-LDS load of row group g (8 rows of 128 bytes, one 16-byte load
// per lane) of a full tile by the calling wave.  While the memory system is
// busy, issuing such a load holds the wave for a while, so a tile's groups are
// spread over all waves and over their compute.
template <typename TX>
__device__ __forceinline__ void dma_group(char* xt, const TX* x, int64_t b, int64_t t0, int d0, int64_t L,
                                          int D, int lane, int g) {
  constexpr int XE = (int)sizeof(TX);
  const int64_t rowb = (int64_t)D * XE;
  const char* src = reinterpret_cast<const char*>(x) + ((b * L + t0) * D + d0) * XE + (int64_t)(8 * g) * rowb;
  // the lane's offset, recomputed here rather than kept live across the loops
  int ln = lane;
  asm volatile("" : "+v"(ln));
  const uint32_t loff = (uint32_t)((ln >> 3) * rowb) + (ln & 7) * 16;
  lds_dma16(src, loff, xt + g * XLay<XE>::GRP);
}

// Row group g of a full output tile from its LDS buffer by the calling wave:
// a 16-byte row store per lane, read from LDS as an 8-byte pair.
template <typename TY>
__device__ __forceinline__ void store_group(TY* y, const char* xt, int64_t b, int64_t t0, int d0, int64_t L,
                                            int D, int lane, int g) {
  constexpr int YE = (int)sizeof(TY);
  const int64_t rowb = (int64_t)D * YE;
  char* dst = reinterpret_cast<char*>(y) + ((b * L + t0) * D + d0) * YE + (int64_t)(8 * g) * rowb;
  int ln = lane;
  asm volatile("" : "+v"(ln));
  const uint32_t loff = (uint32_t)((ln >> 3) * rowb) + (ln & 7) * 16;
  const uint2* s = reinterpret_cast<const uint2*>(xt + g * XLay<YE>::GRP + ln * 16);
  const uint2 u = s[0], w = s[1];
  const u32x4 v = {u.x, u.y, w.x, w.y};
  st_row16(dst, loff, v);
}

// Element copy of a tile that is not full (all threads); zeros outside the tensor.
template <typename TX>
__device__ __forceinline__ void copy_tile(char* xt, const TX* x, int64_t b, int64_t t0, int d0, int64_t L,
                                          int D, int tid) {
  typedef SegGeo<TX> G;
  constexpr int DW = G::DW, XE = (int)sizeof(TX);
  for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
    const int t = idx / DW, c = idx % DW;
    TX v = from_f32<TX>(0.f);
    if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
    *reinterpret_cast<TX*>(xt + XLay<XE>::off(t) + c * XE) = v;
  }
}

// Output tile that is not full, from its LDS buffer (all threads): guarded
// element stores.
template <typename TY>
__device__ __forceinline__ void store_tile_part(TY* y, const char* xt, int64_t b, int64_t t0, int d0, int64_t L,
                                                int D, int tid) {
  typedef SegGeo<TY> G;
  constexpr int DW = G::DW, YE = (int)sizeof(TY);
  for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
    const int t = idx / DW, c = idx % DW;
    if (t0 + t < L && d0 + c < D)
      y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + XLay<YE>::off(t) + c * YE);
  }
}

template <typename TX, typename TY>
__global__ __launch_bounds__(SegGeo<TX>::NT, 1) void fwd_seg_kernel(FwdArgs a) {
  typedef SegGeo<TX> G;
  typedef FPath<TX> PT;
  constexpr int DW = G::DW, NW = G::NW, CW = G::CW, NG = G::NG, NBUF = G::NBUF, XE = (int)sizeof(TX);
  constexpr int NM = fwd_mats(1);  // T, V, U
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) char xb[NBUF][XLay<XE>::BYTES];  // the segment's tile buffers
  // per wave and slot: the chunk states of one channel [component][chunk]
  // (rows of HSTR floats) and, in the 4 spare floats of each row, the block
  // aggregates [component][block]
  constexpr int HSTR = 20;
  constexpr int SLOTS = G::SLOTS;
  __shared__ __align__(16) float s_h[NW][SLOTS][16 * HSTR];
  // per (channel, row q), last tile of a row: the drive part of the state at
  // t = L-1, then the state entering its chunk
  __shared__ __align__(16) f4 s_tail[DW * 4], s_hn[DW * 4];
  __shared__ uint32_t s_tk;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int ln = lane & 15, lq = lane >> 4;                   // chunk, mode pair (2 lq, 2 lq + 1)
  const int nchains = (int)(a.B * a.NB);
  const f4 zero = {0.f, 0.f, 0.f, 0.f}, one = {1.f, 0.f, 1.f, 0.f};
  const char* tab = reinterpret_cast<const char*>(a.tab);
  const int c0 = wave * CW;  // this wave's first channel within the tile

  // segment of the ticket: time-major over the chains, so that every segment's
  // predecessors in its row hold smaller tickets (taken by running work-groups)
  if (tid == 0) s_tk = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int64_t tk = (int64_t)__builtin_amdgcn_readfirstlane(s_tk);
  // a ticket past the last segment means the counter was not reset for this
  // launch: flag it and touch nothing (uniform over the work-group)
  if (tk >= (int64_t)nchains * a.seg_per_chain) {
    if (tid == 0) atomicOr(a.error, 2u);
    return;
  }
  const int64_t seg = tk / nchains;
  const int chain = (int)(tk % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t pb = seg * a.seg_len;                                 // first tile
  const int nt = (int)(a.P - pb < a.seg_len ? a.P - pb : a.seg_len);  // tiles of the segment
  const bool last_seg = (seg == a.seg_per_chain - 1);
  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;

  // the lane's operand rows (the lane offset recomputed at each use rather than
  // kept live in a 64-bit register)
  auto tab_of = [&](int k) {
    int l = lane;
    asm volatile("" : "+v"(l));
    return tab + (size_t)(d0 + c0 + k) * NM * TAB_MAT_BYTES + (uint32_t)l * TAB_LANE_BYTES;
  };
  auto scal_of = [&](int k) { return a.scal + (size_t)(d0 + c0 + k) * a.Mp + 2 * lq; };
  // tiles 0 .. nfull-1 of the segment are full: whole channel block, aligned
  // rows, all TILE_T steps inside the sequence (only a row's last tile can be short)
  const int nfull = __builtin_amdgcn_readfirstlane(
      (a.fast_io && d0 + DW <= a.D) ? ((pb + nt) * TILE_T <= a.L ? nt : nt - 1) : 0);
  auto tile_full = [&](int t) { return t < nfull; };
  // Tile t of the segment into buffer u.  Full tiles go straight to LDS, each
  // wave loading row groups wave, wave + NW, ... (while the memory system is
  // busy, issuing a load holds the wave; spread over all waves, that time is the
  // same for each).  Other tiles are copied by all threads when they are used.
  constexpr int LPT = TILE_T / 8 / NW;  // row groups per wave and tile (loads, stores)
  // this wave's row group i (< LPT) of tile t into buffer u
  auto request_group = [&](int t, int u, int i) {
    if (t < nt && tile_full(t))
      dma_group<TX>(xb[u], reinterpret_cast<const TX*>(a.x), b, (pb + t) * TILE_T, d0, a.L, a.D, lane, wave + NW * i);
  };
  auto request = [&](int t, int u) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) request_group(t, u, i);
  };
  // the row groups a wave issues after its channel k: i with i CW / LPT == k
  auto groups_at = [&](int k, auto&& f) {
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      if ((i * CW) / LPT == k) f(i);
  };
  auto full_in = [&](int lo, int hi) {  // full tiles among lo .. hi
    int n = 0;
    for (int u = lo; u <= hi; ++u) n += tile_full(u) ? 1 : 0;
    return n;
  };
  // Make tile t in buffer u usable: wait for this wave's share of it, or copy
  // it; the caller synchronises.  `later` full tiles have been requested after
  // tile t.  Loads complete in order, so while a load of tile t is pending, so
  // are the LPT * later loads issued after it: vmcnt(LPT * later) waits for
  // tile t exactly (pending stores only raise the count, which errs on the
  // side of waiting).
  auto arrive = [&](int t, int u, int later) {
    if (tile_full(t)) {
      wait_vmcnt(LPT * later);
    } else {
      copy_tile<TX>(xb[u], reinterpret_cast<const TX*>(a.x), b, (pb + t) * TILE_T, d0, a.L, a.D, tid);
    }
  };

  // operands and multipliers first, so that waiting for them waits for no tile
  typename PT::AOp vop[CW];
#pragma unroll
  for (int k = 0; k < CW; ++k) vop[k] = PT::load_a(tab_of(k) + TAB_MAT_BYTES);
  // pass 1 weights: mu^(15-n) of the lane's modes (rows [d][j][Mp] of lambda^(16 j)), lambda^256
  f4 ww[CW], lt[CW];
#pragma unroll
  for (int k = 0; k < CW; ++k) {
    ww[k] = load_f4(a.mpow + ((size_t)(d0 + c0 + k) * CHUNK + (CHUNK - 1 - ln)) * a.Mp + 2 * lq);
    const ModeScalars* ms = scal_of(k);
    lt[k] = mode_pair(ms[0].lamT, ms[1].lamT);
  }
  // Pass 1 visits the tiles last to first, so that tiles 0 .. R-1 (R =
  // min(nt, NBUF)) are the ones still in the buffers when pass 2 starts.  Pass
  // 1's j-th tile (tile nt-1-j) uses buffer j % NBUF; in pass 2 tile t uses
  // buffer (nt-1-(t % NBUF)) % NBUF, which agrees for t < R, and tile t >= R
  // follows tile t - NBUF into its buffer.
  const int R = nt < NBUF ? nt : NBUF;
  auto buf2 = [&](int t) { return (nt - 1 - (t % NBUF)) % NBUF; };
  // block aggregate slot of (channel slot kk, component i): 4 floats
  auto blk = [&](int j, int i) -> float* { return &s_h[wave][j][i * HSTR + 16]; };
  // The operand loads above are complete before the first tile is requested:
  // the compiler does not see the tile loads, and a wait it places for an
  // operand inside the loops would also wait for them.
  __builtin_amdgcn_s_waitcnt(0);
  for (int j = 0; j < NBUF && j < nt; ++j) request(nt - 1 - j, j);

  // ---- pass 1: the segment's own end state ---------------------------------
  // sagg = sum over tiles t and chunks n of lambda^(256 (nt-1-t)) mu^(15-n) S_t[n];
  // lane-wise, with the weight carried from tile to tile (last tile first)
  f4 sagg[CW];
  {
#pragma unroll
    for (int k = 0; k < CW; ++k) sagg[k] = zero;
    for (int j = 0; j < nt; ++j) {
      const int t = nt - 1 - j;
      // visits requested so far: 0 .. NBUF-1, then one more per visit from the second on
      const int last = min((j == 0 ? NBUF - 1 : j + NBUF - 2), nt - 1);
      arrive(t, j % NBUF, full_in(nt - 1 - last, t - 1));
      __syncthreads();  // tile t is in; the buffer of the tile visited before it is free
      // the next request (into the buffer of the tile visited before), spread over the channels
      const bool req = j >= 1 && j + NBUF - 1 < nt;
      const int rt = nt - j - NBUF, ru = (j + NBUF - 1) % NBUF;
      const char* xt = xb[j % NBUF];
#pragma unroll
      for (int gr = 0; gr < NG; ++gr) {
        typename PT::XOp xv[4];
        PT::gather4(xt, c0 + 4 * gr, ln, lq, xv);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int k = 4 * gr + kk;
          sagg[k] = c2fma(ww[k], PT::mma(vop[k], xv[kk], zero), sagg[k]);
          ww[k] = c2mul(ww[k], lt[k]);
          if (req) groups_at(k, [&](int i) { request_group(rt, ru, i); });
        }
      }
      if (pb + t == a.P - 1 && a.h_out != nullptr && ln == nstar) {
        // last tile of the row: sum_{j <= jstar} lambda^(jstar-j) x[16 nstar + j]
        for (int k = 0; k < CW; ++k) {
          const ModeScalars* ms = scal_of(k);
          const f4 lam = mode_pair(ms[0].lam, ms[1].lam);
          f4 tl = zero;
          for (int i = 0; i <= jstar; ++i) {
            const float xr =
                to_f32(*reinterpret_cast<const TX*>(xt + XLay<XE>::off(nstar * CHUNK + i) + (c0 + k) * XE));
            const f4 xin = {xr, 0.f, xr, 0.f};
            tl = c2fma(lam, tl, xin);
          }
          s_tail[(c0 + k) * 4 + lq] = tl;
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < CW; ++k) sagg[k] = row_sum(sagg[k]);

  // ---- the state entering the segment (per wave sub-chain) ----------------------
  // c = lamS^seg h0 + sum_{j<seg} lamS^(seg-1-j) agg_j with lamS = lambda^(256
  // seg_len): term u = seg-1-j (u = seg: h0) goes to lane u % 16 of every row,
  // weighted by lamS^(u % 16) and summed over the row; blocks of 16 terms are
  // combined farthest first by Horner's rule with lamS^16.  The order is fixed
  // by seg alone, so the result is bitwise reproducible.  Payload words start
  // as a signalling-NaN pattern, which arithmetic never produces, so a word
  // that differs from it has been published.
  const int64_t sub = tk * NW + wave;
  // payload of sub-chain s, channel k: 8 modes as float2; the lane's pair at 2 lq
  auto pay = [&](int64_t s, int k) { return ((size_t)s * CW + k) * MODES_PER_GROUP + 2 * lq; };
  // pass 2's T and U operands and chunk multipliers, requested now (ahead of
  // the publishing stores, whose completion later loads of the wave wait for)
  // so that their latency overlaps the wait for the predecessors
  typename PT::AOp top[CW];
  typename PT::UOp uop[CW];
  float2 z1[CW], z4[CW];
#pragma unroll
  for (int k = 0; k < CW; ++k) {
    top[k] = PT::load_a(tab_of(k));
    uop[k] = PT::u_op(load_f4(tab_of(k) + 2 * TAB_MAT_BYTES));
    z1[k] = a.mpow[((size_t)(d0 + c0 + k) * CHUNK + 1) * a.Mp + (ln >> 1)];
    z4[k] = a.mpow[((size_t)(d0 + c0 + k) * CHUNK + 4) * a.Mp + (ln >> 1)];
  }
  if (!last_seg && ln == 0)  // publish this segment's own end state
#pragma unroll
    for (int k = 0; k < CW; ++k) st_agent4(a.pay_agg + pay(sub, k), sagg[k]);
  f4 carry[CW];
  {
    // lamS^n (n the lane's chunk) and lamS^16 of the lane's modes, from the table
    auto spw = [&](int k, int n) {
      return load_f4(a.spow + ((size_t)(d0 + c0 + k) * (CHUNK + 1) + n) * a.Mp + 2 * lq);
    };
#pragma unroll
    for (int k = 0; k < CW; ++k) carry[k] = zero;
    for (int64_t blk = seg / CHUNK; blk >= 0; --blk) {
      const int64_t u = blk * CHUNK + ln;
      const float2* src = a.pay_agg + pay(((seg - 1 - u) * nchains + chain) * NW + wave, 0);
      f4 v[CW];
      for (uint32_t it = 0;; ++it) {
        bool ok = true;
        if (u < seg) {
#pragma unroll
          for (int k = 0; k < CW; ++k) {
            v[k] = ld_agent4(src + (size_t)k * MODES_PER_GROUP);
            ok = ok && __float_as_uint(v[k][0]) != PAY_EMPTY && __float_as_uint(v[k][1]) != PAY_EMPTY &&
                 __float_as_uint(v[k][2]) != PAY_EMPTY && __float_as_uint(v[k][3]) != PAY_EMPTY;
          }
        }
        if (__ballot(!ok) == 0) break;
        if (it >= SPIN_LIMIT) {  // unreachable in ticket order; give up and flag it
          if (lane == 0) atomicOr(a.error, 1u);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
#pragma unroll
      for (int k = 0; k < CW; ++k) {
        if (u >= seg) {
          v[k] = zero;
          if (u == seg && a.h0 != nullptr && d0 + c0 + k < a.D) {
            const float* h = a.h0 + ((size_t)(b * a.D + d0 + c0 + k) * a.M + 2 * lq) * 2;
            if (2 * lq < a.M) v[k][0] = h[0], v[k][1] = h[1];
            if (2 * lq + 1 < a.M) v[k][2] = h[2], v[k][3] = h[3];
          }
        }
        const f4 blk_sum = row_sum(c2mul(spw(k, ln), v[k]));
        // (the farthest block starts from zero)
        carry[k] = blk == seg / CHUNK ? blk_sum : c2fma(spw(k, CHUNK), carry[k], blk_sum);
      }
    }
  }

  // ---- pass 2: the chunk scans and the outputs ----------------------------------
  // S^T = (V x)^T puts component c = ln of chunks 4q .. 4q+3 (q = lq) in lane
  // (c, q); the partner component (re <-> im of the same mode) is in lane c ^ 1.
  // Per tile and channel: block aggregates A_q (Horner over the lane's 4
  // chunks), their exchange through LDS, the block entry states
  // E_{q+1} = mu^4 E_q + A_q from the tile's entering state E_0, the lane's 4
  // chunk states from E_q, and their transpose through LDS into the B operand
  // of y += U H.  A complex factor z acts on a component v with partner p as
  // Re z v + s Im z p, s = -1 for the real part and +1 for the imaginary part.
  float cin[CW], m1r[CW], m1s[CW], m4r[CW], m4s[CW];
  // the entering state as component ln (the fold leaves modes 2 lq, 2 lq + 1 in row lq)
  if (ln == 0)
#pragma unroll
    for (int k = 0; k < CW; ++k) *reinterpret_cast<f4*>(&s_h[wave][0][k * 16 + 4 * lq]) = carry[k];
  wave_lds_order();
#pragma unroll
  for (int k = 0; k < CW; ++k) cin[k] = s_h[wave][0][k * 16 + ln];
  wave_lds_order();
#pragma unroll
  for (int k = 0; k < CW; ++k) {
    vop[k] = PT::load_a(tab_of(k) + TAB_MAT_BYTES);  // (not held through the carry phase)
    const float sgn = (ln & 1) ? 1.f : -1.f;
    m1r[k] = z1[k].x;
    m1s[k] = sgn * z1[k].y;
    m4r[k] = z4[k].x;
    m4s[k] = sgn * z4[k].y;
  }
  // z v + (partner): one complex multiply-add on the lane's component
  auto cstep = [](float zr, float zs, float v, float add) { return cfma_pair(zr, zs, v, add); };
  // At the top of tile t (after the barrier) all threads store tile t-1's
  // outputs from its buffer, and the buffer whose stores were issued one tile
  // earlier (all waves have since passed a barrier, so its LDS reads are done)
  // takes the next tile.  With float32 outputs leaving from the MFMA registers,
  // tile t-1's buffer is free at once.
  constexpr int LAG = SEPY ? 1 : 2;
  static_assert(NBUF > LAG, "a tile is requested before the tile that follows it into its buffer arrives");
  // (pass 2's operands are in registers before its first tile load; the wait
  // also covers the loads of the carry phase)
  __builtin_amdgcn_s_waitcnt(0);
  for (int t = 0; t < nt; ++t) {
    // tiles 0 .. R-1 are still in their buffers from pass 1; before tile t,
    // tiles up to t - 1 - LAG + NBUF have been requested
    if (t >= R) arrive(t, buf2(t), full_in(t + 1, min(t - 1 - LAG + NBUF, nt - 1)));
    __syncthreads();  // tile t is in; tile t-1's outputs are in its buffer
    // tile t-1's stores and the next request, spread over the channels (a tile
    // that is not full is stored here by all threads)
    const bool stf = !SEPY && t >= 1 && tile_full(t - 1);
    if (!SEPY && t >= 1 && !tile_full(t - 1))
      store_tile_part<TY>(reinterpret_cast<TY*>(a.y), xb[buf2(t - 1)], b, (pb + t - 1) * TILE_T, d0, a.L, a.D,
                          tid);
    const bool req = t >= LAG;
    const int rt = t - LAG + NBUF, ru = req ? buf2(t - LAG) : 0;
    auto side = [&](int k) {
      groups_at(k, [&](int i) {
        if (stf)
          store_group<TY>(reinterpret_cast<TY*>(a.y), xb[buf2(t - 1)], b, (pb + t - 1) * TILE_T, d0, a.L, a.D,
                          lane, wave + NW * i);
        if (req) request_group(rt, ru, i);
      });
    };
    char* xt = xb[buf2(t)];
    const int64_t p = pb + t;
#pragma unroll
    for (int gr = 0; gr < NG; ++gr) {
      typename PT::XOp xv[4];
      PT::gather4(xt, c0 + 4 * gr, ln, lq, xv);
      f4 acc[4];
      // y of channel k from its transposed states: lane (n, q) takes components
      // 4q .. 4q+3 of chunk n
      auto apply = [&](int kk, int k, const float* sh) {
        f4 hb;
#pragma unroll
        for (int j = 0; j < 4; ++j) hb[j] = sh[(4 * lq + j) * HSTR + ln];
        acc[kk] = PT::mma_u(uop[k], hb, PT::mma(top[k], xv[kk], zero));
        if (p == a.P - 1 && ln == nstar) s_hn[(c0 + k) * 4 + lq] = hb;  // state entering chunk nstar
      };
      // SLOTS channels at a time: block aggregates (A_q, into the spare
      // columns of the channel's slot), block entry states E_q, chunk entry
      // states (into the slot, transposed on the way out), then y
#pragma unroll
      for (int k0 = 0; k0 < 4; k0 += SLOTS) {
        f4 sk[SLOTS];
#pragma unroll
        for (int j = 0; j < SLOTS; ++j) {
          const int kk = k0 + j, k = 4 * gr + kk;
          sk[j] = PT::mma_t(xv[kk], vop[k], zero);
          float ag = sk[j][0];
#pragma unroll
          for (int r = 1; r < 4; ++r) ag = cstep(m1r[k], m1s[k], ag, sk[j][r]);
          blk(j, ln)[lq] = ag;  // A_lq of component ln
          side(k);
        }
        wave_lds_order();
#pragma unroll
        for (int j = 0; j < SLOTS; ++j) {
          const int kk = k0 + j, k = 4 * gr + kk;
          const f4 A = *reinterpret_cast<const f4*>(blk(j, ln));
          // E_0 = c, E_{q+1} = mu^4 E_q + A_q; E_4 enters the next tile
          float e = cin[k], eq = e;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            e = cstep(m4r[k], m4s[k], e, A[q]);
            if (lq == q + 1) eq = e;
          }
          cin[k] = e;
          // states entering chunks 4 lq .. 4 lq + 3
          f4 h;
          h[0] = eq;
#pragma unroll
          for (int r = 1; r < 4; ++r) h[r] = cstep(m1r[k], m1s[k], h[r - 1], sk[j][r - 1]);
          *reinterpret_cast<f4*>(&s_h[wave][j][ln * HSTR + 4 * lq]) = h;
        }
        wave_lds_order();
#pragma unroll
        for (int j = 0; j < SLOTS; ++j) apply(k0 + j, 4 * gr + k0 + j, s_h[wave][j]);
        wave_lds_order();
      }
      wave_lds_order();
      if (SEPY)
        put_y4_global(reinterpret_cast<float*>(a.y), acc, b, p * TILE_T + ln * CHUNK + lq * 4,
                      d0 + c0 + 4 * gr, a.L, a.D);
      else
        put_y4<TY>(xt, c0 + 4 * gr, ln, lq, acc);
    }
  }
  __syncthreads();  // the last tile's outputs are in its buffer
  if (!SEPY) {
    if (tile_full(nt - 1)) {
#pragma unroll
      for (int i = 0; i < LPT; ++i)
        store_group<TY>(reinterpret_cast<TY*>(a.y), xb[buf2(nt - 1)], b, (pb + nt - 1) * TILE_T, d0, a.L, a.D,
                        lane, wave + NW * i);
    } else {
      store_tile_part<TY>(reinterpret_cast<TY*>(a.y), xb[buf2(nt - 1)], b, (pb + nt - 1) * TILE_T, d0, a.L, a.D,
                          tid);
    }
  }
  if (pb + nt == a.P && a.h_out != nullptr && lane < 4 * CW) {
    // state at t = L-1: lambda^(jstar+1) times the state entering chunk nstar,
    // plus the drive part from pass 1 (the wave's own entries)
    const int k = lane >> 2, r = lane & 3, d = d0 + c0 + k;
    const ModeScalars* ms = a.scal + (size_t)d * a.Mp + 2 * r;
    const f4 hl = c2fma(mode_pair(ms[0].lamTail, ms[1].lamTail), s_hn[(c0 + k) * 4 + r], s_tail[(c0 + k) * 4 + r]);
    if (d < a.D) {
      float* ho = a.h_out + ((size_t)(b * a.D + d) * a.M + 2 * r) * 2;
      if (2 * r < a.M) ho[0] = hl[0], ho[1] = hl[1];
      if (2 * r + 1 < a.M) ho[2] = hl[2], ho[3] = hl[3];
    }
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------
template <typename TA>
hipError_t launch_prep(const Geometry& g, const float* gamma, const float* omega, const float* amp,
                       const float* phase, bool bwd, void* tab, ModeScalars* scal, ModeCarry* cc,
                       hipStream_t st, float2* mpow, float2* spow, uint32_t* flags, int64_t nflags) {
  if (bwd)
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(PREP_THREADS), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, mpow,
                       spow, flags, nflags);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(PREP_THREADS), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, mpow,
                       spow, flags, nflags);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       hipStream_t, float2*, float2*, uint32_t*, int64_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*,
                                        hipStream_t, float2*, float2*, uint32_t*, int64_t);

template <typename TX>
hipError_t launch_fwd_agg(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                          hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    launch_timed(fwd_agg_kernel<TX, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(fwd_agg_kernel<TX, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_agg<float>(const Geometry&, const FwdArgs&, hipStream_t, hipEvent_t,
                                          hipEvent_t);
template hipError_t launch_fwd_agg<bf16_t>(const Geometry&, const FwdArgs&, hipStream_t, hipEvent_t,
                                           hipEvent_t);

hipError_t launch_fwd_carry(const Geometry& g, const FwdArgs& a, hipStream_t st) {
  // segments: at most CARRY_SEG_MAX per row, CARRY_BLOCK * 2^k tiles each
  int seg_len = CARRY_BLOCK;
  while ((g.P + seg_len - 1) / seg_len > CARRY_SEG_MAX) seg_len *= 2;
  const int nseg = (int)((g.P + seg_len - 1) / seg_len);
  int nsegp = 1;
  while (nsegp < nseg) nsegp *= 2;
  const int pw = 256 / nsegp;
  const int pairs_per_tile = g.DW * g.Mp;
  const int64_t npairs = g.B * g.NB * (int64_t)pairs_per_tile;
  const int cpw = g.DW / NWAVES;
  const int pairs_w = (cpw / 4) * g.MG;
  hipLaunchKernelGGL(fwd_carry_kernel, dim3((unsigned)((npairs + pw - 1) / pw)), dim3(256), 0, st, a,
                     seg_len, nseg, nsegp, pairs_per_tile, cpw, pairs_w);
  return hipGetLastError();
}

template <typename TX, typename TY>
hipError_t launch_fwd_segments(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                               hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.NB * a.seg_per_chain)), block(SegGeo<TX>::NT);
  launch_timed(fwd_seg_kernel<TX, TY>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_segments<float, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                      hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_segments<bf16_t, bf16_t>(const Geometry&, const FwdArgs&, hipStream_t,
                                                        hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_segments<bf16_t, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                       hipEvent_t, hipEvent_t);

template <typename TX, typename TY>
hipError_t launch_fwd_apply(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    launch_timed(fwd_apply_kernel<TX, TY, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(fwd_apply_kernel<TX, TY, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_apply<float, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                   hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_apply<bf16_t, bf16_t>(const Geometry&, const FwdArgs&, hipStream_t,
                                                     hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_apply<bf16_t, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                    hipEvent_t, hipEvent_t);

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace res
