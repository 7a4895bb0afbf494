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
#include "stream.h"
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
                                                   int MG, int last_len,
                                                   TA* __restrict__ tab,
                                                   ModeScalars* __restrict__ scal,
                                                   ModeCarry* __restrict__ cc) {
  // lambda^0..16, then lambda^128, lambda^256, lambda^last_len
  constexpr int NPW = CHUNK + 1 + 3;
  const int d = blockIdx.x;
  const int Mp = MODES_PER_GROUP * MG;
  __shared__ double2 pw[MODES_PER_GROUP * MG_MAX][NPW];
  __shared__ double2 cm[MODES_PER_GROUP * MG_MAX];  // c
  __shared__ double2 ep[MODES_PER_GROUP * MG_MAX];  // e^{i phase}
  __shared__ double taps[CHUNK + 1];

  const bool dvalid = d < D;
  // one round: the table powers and c
  const int n_pw = Mp * (NPW + 1);
  for (int t = threadIdx.x; t < n_pw; t += blockDim.x) {
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
      double2 z = make_double2(0.0, 0.0), e = z;
      if (valid) {
        double sn, cs;
        sincos((double)phase[d * M + m], &sn, &cs);
        const double av = (double)amp[d * M + m];
        z = make_double2(av * cs, av * sn);
        e = make_double2(cs, sn);
      }
      cm[m] = z;
      ep[m] = e;
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
    mc.lam1 = lam;
    mc.c = cm[m];
    mc.ephi = ep[m];
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
    const int g = (mat - 1) / 3, s = (mat - 1) % 3;
    const int mi = g * 8 + i / 2;
    switch (s) {
      case 0: return part(pw[mi][k], i & 1);                      // Eq[comp i][k] = lambda^k
      case 1: return k * part(pw[mi][k], i & 1);                  // Er = k lambda^k
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
  // every thread of a (row, pair) has read h0 before the last segment's thread
  // writes h_out below, so h_out may be the h0 buffer
  __syncthreads();
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
// Single-pass forward (one mode group, M <= 8).
//
// A chain is one batch row and one block of DW channels (128-byte rows).  The G
// work-groups that serve a chain cut it into G contiguous segments of tiles
// (256 steps).  On arrival a work-group counts itself in the chain; once all G
// have arrived (they are then all running) the work-group of rank r (block
// index over the number of chains) takes segment r.  If they do not all arrive
// within a short bounded wait (part of the device is busy with other work), the
// chain hands out its segments by ticket instead, first come first served, so
// that every segment a look-back waits for belongs to a running work-group.
//   tables   built in LDS by the work-group itself while its first tile loads;
//            each wave keeps its channels' T, V, U operands in registers.
//   phase A  the segment's tiles, last to first: per channel S = V x on MFMA
//            (lane (c, q): component c of chunks 4q .. 4q+3); lane swaps leave
//            component c of channel k in lane (c, k) for all 16 chunks; the
//            tile's end state from a zero start, A = sum_n mu^(15-n) S[n]
//            (mu = lambda^16), is 16 steps A <- mu A + S[n] in the lane's own
//            registers, and the segment's Aseg = sum_k lambda^(256 k) A of its
//            k-th last tile.  The first three tiles stay in LDS.
//   look-back  the segment publishes P_j (segment 0: its inclusive end state
//            from h0; the others: Aseg), then folds the published P_i of the
//            earlier segments, oldest first, E <- lambda^(256 S_i) E + P_i.
//   phase B  the segment's tiles in order: H[0] = E, H[n+1] = mu H[n] + S[n]
//            (the same 16 steps), moved through LDS into the MFMA operand layout;
//            y = T x + U H is rounded into the tile buffer and leaves as 128-byte
//            rows; E moves on as the scan's end state.
// Every wave issues its share of the tile loads (direct to LDS) and row stores.
// A published state is a set of 64-bit device-coherent words, each a float and
// the call's tag, so a reader checks the data itself; the counters are reset by
// the last work-group of a chain to finish.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t ld_flag(const uint32_t* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(uint32_t* f, uint32_t v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Upper bound on polls of one wait for a published state (with a short sleep
// between polls, well over 0.1 s).  Every such wait ends long before it; it is
// reached only with a workspace that was not zeroed before its first use (or was
// changed meanwhile): the kernel then records bit 0 in the status word and goes on.
constexpr uint32_t SPIN_LIMIT = 1u << 18;
// Polls of the wait for the other work-groups of a chain to arrive (some tens of
// microseconds at most); past it the chain takes its tiles by ticket.
constexpr uint32_t ARRIVE_WAIT = 64;
#ifndef RES_FOLD_WORDS
#define RES_FOLD_WORDS 16
#endif

// Direct-to-LDS load of row group g (8 rows of 128 bytes, one 16-byte load
// per lane) of a full tile by the calling wave.
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

// Row groups g0, g0 + step, ... (n of them) of a full output tile from its LDS
// buffer by the calling wave: all the LDS reads first (a 16-byte row piece per
// lane, read as two 8-byte halves), then the 16-byte row stores.
template <typename TY, int N>
__device__ __forceinline__ void store_groups(TY* y, const char* xt, int64_t b, int64_t t0, int d0, int64_t L,
                                             int D, int lane, int g0, int step) {
  constexpr int YE = (int)sizeof(TY);
  const int64_t rowb = (int64_t)D * YE;
  char* dst = reinterpret_cast<char*>(y) + ((b * L + t0) * D + d0) * YE;
  int ln = lane;
  asm volatile("" : "+v"(ln));
  u32x4 v[N];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint2* s = reinterpret_cast<const uint2*>(xt + (g0 + step * i) * XLay<YE>::GRP + ln * 16);
    const uint2 u = s[0], w = s[1];
    v[i] = u32x4{u.x, u.y, w.x, w.y};
  }
  const uint32_t loff = (uint32_t)((ln >> 3) * rowb) + (ln & 7) * 16;
#pragma unroll
  for (int i = 0; i < N; ++i) st_row16(dst + (int64_t)(8 * (g0 + step * i)) * rowb, loff, v[i]);
}

// Element copy of a tile that is not full (NT threads); zeros outside the tensor.
template <typename TX, int NT>
__device__ __forceinline__ void copy_tile(char* xt, const TX* x, int64_t b, int64_t t0, int d0, int64_t L,
                                          int D, int tid) {
  constexpr int DW = tile_channels<TX>(), XE = (int)sizeof(TX);
  for (int idx = tid; idx < TILE_T * DW; idx += NT) {
    const int t = idx / DW, c = idx % DW;
    TX v = from_f32<TX>(0.f);
    if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
    *reinterpret_cast<TX*>(xt + XLay<XE>::off(t) + c * XE) = v;
  }
}

// Output tile that is not full, from its LDS buffer (NT threads): guarded
// element stores.
template <typename TY, int NT>
__device__ __forceinline__ void store_tile_part(TY* y, const char* xt, int64_t b, int64_t t0, int d0, int64_t L,
                                                int D, int tid) {
  constexpr int DW = tile_channels<TY>(), YE = (int)sizeof(TY);
  for (int idx = tid; idx < TILE_T * DW; idx += NT) {
    const int t = idx / DW, c = idx % DW;
    if (t0 + t < L && d0 + c < D)
      y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + XLay<YE>::off(t) + c * YE);
  }
}

template <typename TX>
struct StreamGeo {
  static constexpr int DW = tile_channels<TX>();   // channels per tile: 64 (bf16) | 32 (float)
  static constexpr int NW = 8;                     // waves (two per SIMD: 256 registers each)
  static constexpr int NG = DW / (4 * NW);         // groups of 4 channels per wave: 2 | 1
  static constexpr int NT = 64 * NW;
  static constexpr int NQ = 0;                     // first load wave
  static constexpr int LW = NW;                    // load waves (every wave loads and stores rows)
  static constexpr int GPL = (TILE_T / 8) / LW;    // row groups per load wave and tile
  static constexpr int NBUF = 4;                   // tile buffers
  static constexpr int HKS = 16 * 16 + 8;          // floats per channel in the H transposition (8 of bank offset)
  static constexpr int XB = XLay<(int)sizeof(TX)>::BYTES;
  static constexpr int HB = NW * 4 * HKS * 4;      // every wave's 4 channels of one group
  static constexpr int BUFB = XB > HB ? XB : HB;   // bytes per buffer (tile, or H transposition)
  static_assert(GPL * LW == TILE_T / 8, "the load waves cover a tile");
  static_assert(NQ + LW <= NW, "control and load waves are distinct");
  static_assert(NG * 4 * NW == DW, "the waves cover the tile's channels");
};

// LDS stage of a work-group's tables, per channel k of the block and mode m:
// lambda^j (j = 0 .. 16) and c as float2, the taps K[tau] (tau = 0 .. 15) as
// float32 or as a bf16 pair (high | low << 16).
template <typename TX>
struct TabStage {
  static constexpr int DW = tile_channels<TX>();
  static constexpr int PW = 0;                     // float2 [DW][8][17]
  static constexpr int CM = PW + DW * 8 * 17 * 8;  // float2 [DW][8]
  static constexpr int TAP = CM + DW * 8 * 8;      // uint32 [DW][16]
  static constexpr int BYTES = TAP + DW * 16 * 4;
};

// Per (channel, mode) constants a work-group keeps in LDS for the whole call
// (each is needed once per tile or less): lambda, lambda^(jstar+1) (the
// terminal state), the segment hops lambda^(256 n) and lambda^(256 (n + 1)) as
// (Re, Im), and lambda^256 in float64 (the powers over a segment).
struct KConst {
  double2 l256;
  float2 lam1, lamt, hop0, hop1;
};

// A float64 moved across lanes by a DPP pattern (its two halves).
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, 0xF, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, (uint64_t)lo | ((uint64_t)hi << 32));
}

// The float32 parameters of thread (k, m) = 8 k + m: channel d0 + k, mode m
// (zeros outside D x M and for threads beyond the block's channels).
struct ModeIn {
  float gamma, omega, amp, phase;
};
template <typename TX>
__device__ __forceinline__ ModeIn load_mode(const StreamArgs& a, int d0, int tid) {
  ModeIn r{0.f, 0.f, 0.f, 0.f};
  const int k = tid >> 3, m = tid & 7, d = d0 + k;
  if (tid < TabStage<TX>::DW * 8 && d < a.D && m < a.M) {
    const int i = d * a.M + m;
    r.gamma = a.gamma[i];
    r.omega = a.omega[i];
    r.amp = a.amp[i];
    r.phase = a.phase[i];
  }
  return r;
}

// The tables of channels d0 .. d0+DW-1 into the stage st (threads (k, m) =
// 8 k + m, one per channel and mode, with their parameters pin).  lambda =
// exp(-gamma) (cos omega, sin omega) and c = amp (cos phase, sin phase) in
// float64, the powers lambda^j by successive products and lambda^256 by eight
// squarings and the segment hops by binary powering of it (a relative error of
// a few 2^-53 per product); the taps
// K[tau] = Re sum_m c lambda^tau, summed in float64 over the eight mode lanes of
// a channel, are rounded once.
template <typename TX>
__device__ void build_tables(const StreamArgs& a, int d0, char* st, KConst* kc, int tid, const ModeIn& pin,
                             int64_t seg) {
  typedef TabStage<TX> S;
  if (tid >= S::DW * 8) return;
  const int k = tid >> 3, m = tid & 7, d = d0 + k;
  double2 z = make_double2(0.0, 0.0), cz = z;
  if (d < a.D && m < a.M) {
    double sn, cs;
    sincos((double)pin.omega, &sn, &cs);
    const double e = exp(-(double)pin.gamma);
    z = make_double2(e * cs, e * sn);
    sincos((double)pin.phase, &sn, &cs);
    const double av = (double)pin.amp;
    cz = make_double2(av * cs, av * sn);
  }
  float2* pw = reinterpret_cast<float2*>(st + S::PW) + tid * 17;
  double tp[16];
  double2 pj = make_double2(1.0, 0.0);
#pragma unroll
  for (int j = 0; j <= 16; ++j) {
    pw[j] = make_float2((float)pj.x, (float)pj.y);
    if (j < 16) tp[j] = cz.x * pj.x - cz.y * pj.y;
    if (j < 16) pj = zmul(pj, z);
  }
  double2 l2 = z;
#pragma unroll
  for (int s = 0; s < 8; ++s) l2 = zmul(l2, l2);
  // the segment hops (lambda^256)^seg and (lambda^256)^(seg+1) by binary powering
  double2 zs0 = make_double2(1.0, 0.0);
  {
    double2 sq = l2;
    for (int64_t e = seg; e > 0; e >>= 1) {
      if (e & 1) zs0 = zmul(zs0, sq);
      sq = zmul(sq, sq);
    }
  }
  const double2 zs1 = zmul(zs0, l2);
  reinterpret_cast<float2*>(st + S::CM)[tid] = make_float2((float)cz.x, (float)cz.y);
  {
    KConst c;
    c.l256 = l2;
    c.lam1 = make_float2((float)z.x, (float)z.y);
    c.lamt = pw[(a.last_len - 1) % CHUNK + 1];
    c.hop0 = make_float2((float)zs0.x, (float)zs0.y);
    c.hop1 = make_float2((float)zs1.x, (float)zs1.y);
    kc[tid] = c;
  }
  // sum over the 8 mode lanes of the channel, halving the taps at each of three
  // exchanges (DPP moves of the two halves of a float64): lane m <-> 7-m keeps
  // taps 0..7 (m < 4) or 8..15, then lane m <-> m^2 keeps a half of those by bit
  // 1 of m, then m <-> m^1 by bit 0; lane m ends with the full sums of taps
  // tau0 and tau0 + 1, tau0 = 8 [m >= 4] + 4 bit1(m) + 2 bit0(m)
  double t8[8], t4[4], t2[2];
  {
    const bool h = m >= 4, b1 = (m >> 1) & 1, b0 = m & 1;
#pragma unroll
    for (int i = 0; i < 8; ++i) t8[i] = (h ? tp[8 + i] : tp[i]) + dpp_f64<0x141>(h ? tp[i] : tp[8 + i]);
#pragma unroll
    for (int i = 0; i < 4; ++i) t4[i] = (b1 ? t8[4 + i] : t8[i]) + dpp_f64<0x4E>(b1 ? t8[i] : t8[4 + i]);
#pragma unroll
    for (int i = 0; i < 2; ++i) t2[i] = (b0 ? t4[2 + i] : t4[i]) + dpp_f64<0xB1>(b0 ? t4[i] : t4[2 + i]);
  }
  {
    const int tau0 = (m >= 4 ? 8 : 0) + ((m >> 1) & 1) * 4 + (m & 1) * 2;
    uint32_t* tap = reinterpret_cast<uint32_t*>(st + S::TAP) + k * 16 + tau0;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (sizeof(TX) == 4) {
        tap[j] = __float_as_uint((float)t2[j]);
      } else {
        const bf16_t hi = from_f32<bf16_t>((float)t2[j]);
        const bf16_t lo = from_f32<bf16_t>((float)(t2[j] - (double)to_f32(hi)));
        tap[j] = (uint32_t)hi | ((uint32_t)lo << 16);
      }
    }
  }
}

// Lane (i, q)'s operands of channel k of the stage, as the MFMA lanes read them:
// T[i][4q+r] = K[i - 4q - r] (zero above the diagonal); V[i][4q+r] = Re or Im
// (by the parity of i) of lambda^(15 - 4q - r) of mode i/2; U[i][4q+r] = Re or
// -Im (by the parity of r) of c lambda^(i+1) of mode (4q + r)/2, formed in
// float32 from the staged float32 power and c.  For bf16 activations T and V are
// split into bf16 halves (high, low).
template <typename TX>
__device__ __forceinline__ void stage_operands(const char* st, int k, int i, int q, typename FPath<TX>::AOp& t,
                                               typename FPath<TX>::AOp& v, f4& u) {
  typedef TabStage<TX> S;
  const float2* pw = reinterpret_cast<const float2*>(st + S::PW) + k * 8 * 17;
  const float2* cm = reinterpret_cast<const float2*>(st + S::CM) + k * 8;
  const uint32_t* tap = reinterpret_cast<const uint32_t*>(st + S::TAP) + k * 16;
  uint32_t tw[4];
  f4 vv;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int kk = 4 * q + r;
    tw[r] = i >= kk ? tap[i - kk] : 0u;
    const float2 pv = pw[(i >> 1) * 17 + 15 - kk];
    vv[r] = (i & 1) ? pv.y : pv.x;
    const float2 c = cm[kk >> 1], pu = pw[(kk >> 1) * 17 + i + 1];
    u[r] = (r & 1) ? -fmaf(c.x, pu.y, c.y * pu.x) : fmaf(c.x, pu.x, -c.y * pu.y);
  }
  if (sizeof(TX) == 4) {
    t = FPath<TX>::load_a_u4(make_uint4(tw[0], tw[1], tw[2], tw[3]));
    v = FPath<TX>::load_a_u4(make_uint4(__float_as_uint(vv[0]), __float_as_uint(vv[1]), __float_as_uint(vv[2]),
                                        __float_as_uint(vv[3])));
  } else {
    uint32_t vh[4], vl[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const bf16_t h = from_f32<bf16_t>(vv[r]);
      vh[r] = h;
      vl[r] = from_f32<bf16_t>(vv[r] - to_f32(h));
    }
    t = FPath<TX>::load_a_u4(make_uint4((tw[0] & 0xFFFFu) | (tw[1] << 16), (tw[2] & 0xFFFFu) | (tw[3] << 16),
                                        (tw[0] >> 16) | (tw[1] & 0xFFFF0000u), (tw[2] >> 16) | (tw[3] & 0xFFFF0000u)));
    v = FPath<TX>::load_a_u4(make_uint4(vh[0] | (vh[1] << 16), vh[2] | (vh[3] << 16), vl[0] | (vl[1] << 16),
                                        vl[2] | (vl[3] << 16)));
  }
}

// S = V x of a wave's four channels (xv: their activation operands), moved so
// that lane (c, k) holds component c of channel k, chunk n in S[n].  The MFMA
// leaves component c of chunks 4q .. 4q+3 of channel k in lane (c, q) of R[k];
// exchanging rows of 16 lanes between the four results (two 32-lane and two
// 16-lane swaps per register) gives lane (c, q) of R[j] the chunks 4j .. 4j+3
// of channel q.
template <typename TX>
__device__ __forceinline__ void chunk_states(const typename FPath<TX>::XOp (&xv)[4],
                                             const typename FPath<TX>::AOp (&vop)[4], float (&S)[16]) {
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  f4 R[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) R[k] = FPath<TX>::mma_t(xv[k], vop[k], zero);
  lanes_to_chunks(R, S);
}

// Published tile end states: every 64-bit word holds one float (low half) and
// the tag of the call that wrote it (high half), so that a reader checks the
// data itself and a writer needs no ordering between data and a flag.  The
// stores and loads are device-coherent (work-groups of a chain run on any XCD).
template <int NG>
__device__ __forceinline__ void put_state(uint64_t* p, const float (&v)[NG], uint32_t tag) {
#pragma unroll
  for (int g = 0; g < NG; ++g)
    __hip_atomic_store(p + g, (uint64_t)__float_as_uint(v[g]) | ((uint64_t)tag << 32), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
// false while any word still carries another tag
template <int NG>
__device__ __forceinline__ bool get_state(const uint64_t* p, uint32_t tag, float (&v)[NG]) {
  bool ok = true;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const uint64_t w = __hip_atomic_load(p + g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    v[g] = __uint_as_float((uint32_t)w);
    ok = ok && (uint32_t)(w >> 32) == tag;
  }
  return ok;
}

template <typename TX, typename TY>
__global__ __launch_bounds__(StreamGeo<TX>::NT, 1) void fwd_stream_kernel(StreamArgs a) {
  typedef StreamGeo<TX> G;
  typedef FPath<TX> PT;
  typedef TabStage<TX> TS;
  constexpr int DW = G::DW, NW = G::NW, NG = G::NG, NT = G::NT, NQ = G::NQ, LW = G::LW, GPL = G::GPL;
  constexpr int NBUF = G::NBUF, XE = (int)sizeof(TX), HKS = G::HKS;
  static_assert(TS::BYTES <= (NBUF - 1) * G::BUFB, "the table stage fits in buffers 1 .. NBUF-1");
  static_assert(NBUF == 4, "buffer rotation assumes four buffers");
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  // published states loaded at a time by the look-back (a register budget of 2 RES_FOLD_WORDS)
  constexpr int FB = RES_FOLD_WORDS / NG;
  __shared__ __align__(16) char xb[NBUF][G::BUFB];
  __shared__ KConst s_kc[DW * 8];
  __shared__ uint32_t s_u[4];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 15, lq = lane >> 4;  // MFMA lane (i, q); scan lane (component ln, channel lq)
  const int cb = wave * 4 * NG;              // this wave's first channel; group g: cb + 4 g .. cb + 4 g + 3
  const bool is_ld = wave >= NQ && wave < NQ + LW;
  const int chain = (int)(blockIdx.x % (unsigned)a.nchains);
  const int64_t b = chain / a.NB;
  const int blk = chain % a.NB;
  const int d0 = blk * DW;
  const int64_t P = a.P;
  const uint32_t G_ = gridDim.x / (uint32_t)a.nchains;  // work-groups (segments) of each chain
  // (channel, mode) of scan lane (component ln, channel lq) of group g
  auto kmode = [&](int g) { return (cb + 4 * g + lq) * 8 + (ln >> 1); };
  // segment j: tiles [j Sf + min(j, Sr), ... + Sf + (j < Sr))
  const int64_t Sf = P / G_, Sr = P % G_;
  auto seg_start = [&](int64_t j) { return j * Sf + (j < Sr ? j : Sr); };
  uint32_t* cw = a.chainw + 4 * (size_t)chain;  // [0] next ticket, [1] arrived, [2] order, [3] finished
  const uint32_t ep = ld_flag(a.hdr + 1);
  const uint32_t TAG = ep + 1u;
  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  const bool full_block = a.fast_io && d0 + DW <= a.D;
  auto tile_full = [&](int64_t p) { return full_block && (p + 1) * TILE_T <= a.L; };
  auto load_tile = [&](int u, int64_t p) {  // by the load waves, a full tile
#pragma unroll
    for (int i = 0; i < GPL; ++i)
      dma_group<TX>(xb[u], reinterpret_cast<const TX*>(a.x), b, p * TILE_T, d0, a.L, a.D, lane,
                    (wave - NQ) + LW * i);
  };
  auto store_tile = [&](int u, int64_t p) {  // rows of output tile p from buffer u
    if (tile_full(p)) {
      if (is_ld) {
        constexpr int SB = GPL < 4 ? GPL : 4;  // row groups per batch of LDS reads
#pragma unroll
        for (int i = 0; i < GPL; i += SB)
          store_groups<TY, SB>(reinterpret_cast<TY*>(a.y), xb[u], b, p * TILE_T, d0, a.L, a.D, lane,
                               (wave - NQ) + LW * i, LW);
      }
    } else {
      store_tile_part<TY, NT>(reinterpret_cast<TY*>(a.y), xb[u], b, p * TILE_T, d0, a.L, a.D, tid);
    }
  };
  // this lane's words of the published aggregate of segment j
  auto a_slot = [&](int64_t j) { return a.agg + ((((size_t)chain * G_ + j) * NW + wave) * 64 + lane) * NG; };

  // ---- arrival, the first tile, the tables ----------------------------------
  // In static order the j-th work-group of a chain by block index takes segment
  // j (static order is chosen only once all G have arrived).  Its segment's last
  // tile loads at once (again below if the chain takes tickets); the arrival
  // count and a first look at the chain's arrivals come back while the tables
  // are built.
  const uint32_t rank = blockIdx.x / (uint32_t)a.nchains;
  const ModeIn pin = load_mode<TX>(a, d0, tid);  // before any tile load of the wave
  uint32_t arr = 0, arrived = 0;
  if (tid == 0) {
    arr = atomicAdd(cw + 1, 1u);
    arrived = ld_flag(cw + 1);
  }
  // With one work-group per chain there is no aggregate to publish (phase A is
  // skipped) and the chain's first tile loads at once.
  const bool phaseA = G_ > 1;
  {
    const int64_t e0 = phaseA ? seg_start(rank + 1) - 1 : 0;
    if (is_ld && tile_full(e0)) load_tile(0, e0);
  }
  char* stg = xb[1];  // the tables are staged in buffers 1 .. 3
  build_tables<TX>(a, d0, stg, s_kc, tid, pin, Sf);
  // ---- the order of the chain's segments: static once every work-group of the
  // chain has arrived, else by ticket; the first CAS decides for the chain (its
  // answer is read after the operands are formed).  More arrivals than
  // work-groups: the counters were not in their initial state (workspace not
  // zeroed, or changed meanwhile); such a work-group touches nothing. ----------
  uint32_t order_old = 0, order_want = 0;
  if (tid == 0) {
    if (arr >= G_) {
      atomicOr(a.hdr, 2u);
      order_want = 0;  // stale
    } else {
      bool all = arrived >= G_;
      for (uint32_t n = 0; !all && n < ARRIVE_WAIT; ++n) {
        __builtin_amdgcn_s_sleep(2);
        all = ld_flag(cw + 1) >= G_;
      }
      order_want = all ? 1u : 2u;
      order_old = atomicCAS(cw + 2, 0u, order_want);
    }
  }
  __syncthreads();
  typename PT::AOp vop[NG][4], top[NG][4];
  typename PT::UOp uop[NG][4];
  // mu = lambda^16 of scan lane (component ln, channel lq of group g), as
  // (Re, -+Im): the re lane keeps -Im, the im lane +Im (cfma_pair)
  const float sgn = (ln & 1) ? 1.f : -1.f;
  auto lane_c = [&](float2 z) { return make_float2(z.x, sgn * z.y); };
  float mur[NG], mus[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f4 uu;
      stage_operands<TX>(stg, cb + 4 * g + k, ln, lq, top[g][k], vop[g][k], uu);
      uop[g][k] = PT::u_op(uu);
    }
    const float2 mu = reinterpret_cast<const float2*>(stg + TS::PW)[kmode(g) * 17 + 16];
    mur[g] = mu.x;
    mus[g] = sgn * mu.y;
  }
  if (tid == 0) {
    const uint32_t order = order_want == 0 ? 0u : order_old == 0 ? order_want : order_old;
    const uint32_t seg = order == 1 ? rank : order == 2 ? atomicAdd(cw, 1u) : 0u;
    // a ticket past the chain's segments: the counters were not in their initial
    // state either
    const bool stale = order == 0 || seg >= G_;
    if (stale && order != 0) atomicOr(a.hdr, 2u);
    s_u[2] = stale ? 0u : order;
    s_u[0] = seg;
  }
  // every earlier vector memory operation of the wave has completed (the first
  // tile among them)
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  if (s_u[2] == 0) return;  // stale counters
  const bool by_ticket = s_u[2] != 1;
  const int64_t j = s_u[0];         // this work-group's segment
  const int64_t s = seg_start(j);   // its first tile
  const int S = (int)(seg_start(j + 1) - s);  // its tiles
  // ---- phase A: the segment's tiles from last to first, k-th into buffer k & 3;
  // its aggregate Aseg = sum_t lambda^(256 (e-1-t)) A_t, A_t the tile's end state
  // from a zero start.  The first three tiles of the segment stay in their
  // buffers; the fourth's buffer is left free for phase B. ---------------------
  uint32_t issued = 0, mark[NBUF] = {0, 0, 0, 0};
  auto tileA = [&](int k) { return s + S - 1 - k; };
  if (!phaseA && is_ld) {
    // phase B's first tiles in buffers 0, 1, 2 (the first loaded above)
#pragma unroll
    for (int k = 1; k < 3; ++k) {
      if (k < S && tile_full(s + k)) {
        load_tile(k, s + k);
        issued += GPL;
      }
      mark[k] = issued;
    }
  }
  if (phaseA && is_ld) {
    // the segment's last tile is in buffer 0 unless the segment came by ticket
    mark[0] = 0;
    if (by_ticket && tile_full(tileA(0))) {
      load_tile(0, tileA(0));
      issued += GPL;
      mark[0] = issued;
    }
#pragma unroll
    for (int k = 1; k < 3; ++k) {
      if (k < S && tile_full(tileA(k))) {
        load_tile(k, tileA(k));
        issued += GPL;
      }
      mark[k] = issued;
    }
  }
  float Aseg[NG];
  double2 pw[NG];  // lambda^(256 k), float64
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    Aseg[g] = 0.f;
    pw[g] = make_double2(1.0, 0.0);
  }
  for (int k = 0; phaseA && k < S; ++k) {
    const int u = k & (NBUF - 1);
    const int64_t p = tileA(k);
    if (tile_full(p)) {
      if (is_ld) wait_vmcnt((int)(issued - mark[u]));
    } else {
      copy_tile<TX, NT>(xb[u], reinterpret_cast<const TX*>(a.x), b, p * TILE_T, d0, a.L, a.D, tid);
    }
    __syncthreads();
    // the tile three ahead, into the buffer of the previous one (read by every
    // wave before this barrier): the first half of the waves issues its loads
    // before pass 1, the other half after it
    auto memory = [&]() {
      const int u3 = (k + 3) & (NBUF - 1);
      if (k + 3 < S && tile_full(tileA(k + 3))) {
        load_tile(u3, tileA(k + 3));
        issued += GPL;
      }
      mark[u3] = issued;
    };
    const bool mem_first = wave < NW / 2;
    if (mem_first) memory();
    const char* xt = xb[u];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      typename PT::XOp xv[4];
      float S16[16];
      PT::gather4(xt, cb + 4 * g, ln, lq, xv);
      chunk_states<TX>(xv, vop[g], S16);
      float A = S16[0];
#pragma unroll
      for (int n = 1; n < 16; ++n) A = cfma_pair(mur[g], mus[g], A, S16[n]);
      // Aseg += lambda^(256 k) A; then the power moves one tile on
      Aseg[g] = cfma_pair((float)pw[g].x, sgn * (float)pw[g].y, A, Aseg[g]);
      pw[g] = zmul(pw[g], s_kc[kmode(g)].l256);
    }
    if (!mem_first) memory();
  }

  // ---- look-back: the state entering the segment, E, from the published states
  // of the chain's earlier segments, oldest first, E <- lambda^(256 S_i) E + P_i.
  // Segment 0 alone reads h0 and publishes its inclusive end state
  // P_0 = lambda^(256 S_0) h0 + Aseg_0; every other segment publishes P_j = Aseg_j.
  // (h0 is then read before anything the chain's last tile waits for, so h_out
  // may be h0's memory.) ----------------------------------------------------------
  float E[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    E[g] = 0.f;
    const int d = d0 + cb + 4 * g + lq, m = ln >> 1;
    if (j == 0 && a.h0 != nullptr && d < a.D && m < a.M)
      E[g] = a.h0[((size_t)(b * a.D + d) * a.M + m) * 2 + (ln & 1)];
  }
  if (G_ > 1) {
    float Pj[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const float2 z = lane_c(Sr > 0 ? s_kc[kmode(g)].hop1 : s_kc[kmode(g)].hop0);  // segment 0's hop
      Pj[g] = j == 0 ? cfma_pair(z.x, z.y, E[g], Aseg[g]) : Aseg[g];
    }
    put_state<NG>(a_slot(j), Pj, TAG);
  }
  bool ok = true;
  for (int64_t q = 0; ok && q < j; q += FB) {
    float Aq[FB][NG];
    for (uint32_t n = 0;; ++n) {
      bool mine = true;
#pragma unroll
      for (int i = 0; i < FB; ++i) mine = get_state<NG>(a_slot(q + i < j ? q + i : q), TAG, Aq[i]) && mine;
      if (__ballot(!mine) == 0) break;
      if (n >= SPIN_LIMIT || ((n & 63) == 63 && ld_flag(a.hdr + 4) != 0)) {
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (!ok) break;
#pragma unroll
    for (int i = 0; i < FB; ++i) {
      if (q + i < j) {
        const bool longer = q + i < Sr;  // segment q+i has Sf + 1 tiles
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          const float2 z = lane_c(longer ? s_kc[kmode(g)].hop1 : s_kc[kmode(g)].hop0);
          E[g] = cfma_pair(z.x, z.y, E[g], Aq[i][g]);
        }
      }
    }
  }
  if (!ok && lane == 0) {  // gave up: the outputs of this call are wrong
    atomicOr(a.hdr, 1u);
    atomicOr(a.hdr + 4, 1u);
  }

  // ---- phase B: the segment's tiles in order, E moving from tile to tile as the
  // scan's end state.  The states H go through one fixed buffer (the one phase A
  // left free, or buffer 3); tiles rotate through the other three: tile s+m is
  // in buffer U[m mod 3], the first three as phase A left them (or as loaded
  // above), each later one loaded into the buffer of the tile three before it
  // once that tile's rows have been read out.  Iteration m: the tile's arrival
  // and one barrier, the load of tile s+m+1, the rows of tile s+m-1 (read out of
  // LDS while pass 2 runs), pass 2 of tile s+m. ---------------------------------
  const int U0 = phaseA ? (S - 1) & 3 : 0, U1 = phaseA ? (S - 2) & 3 : 1, U2 = phaseA ? (S - 3) & 3 : 2;
  const int UH = phaseA ? S & 3 : 3;
  auto ubuf = [&](int m) {
    const int r = m % 3;
    return r == 0 ? U0 : r == 1 ? U1 : U2;
  };
  float* hs = reinterpret_cast<float*>(xb[UH]) + wave * 4 * HKS;
  const int resident = phaseA ? 3 : 0;  // tiles left in their buffers by phase A
  for (int m = 0; m < S; ++m) {
    const int64_t p = s + m;
    const int u = ubuf(m);
    if (m >= resident) {
      if (tile_full(p)) {
        if (is_ld) wait_vmcnt((int)(issued - mark[u]));
      } else {
        copy_tile<TX, NT>(xb[u], reinterpret_cast<const TX*>(a.x), b, p * TILE_T, d0, a.L, a.D, tid);
      }
    }
    // the tile is in; the rows of tile s+m-2 have been read out of its buffer;
    // every wave is done with H and with the outputs of tile s+m-1
    __syncthreads();
    // the rows of tile s+m-1 and the load of tile s+m+1: the first half of the
    // waves issues them before pass 2, the other half after it, so that on
    // every SIMD one wave computes while the other issues its memory operations
    const int un = ubuf(m + 1), up = ubuf(m + 2);  // ubuf(m - 1) == ubuf(m + 2)
    auto memory = [&]() {
      if (!SEPY && m >= 1) {
        store_tile(up, p - 1);
        if (tile_full(p - 1)) issued += GPL;
      }
      if (m + 1 >= 3 && m + 1 < S) {
        if (tile_full(p + 1)) {
          load_tile(un, p + 1);
          issued += GPL;
        }
        mark[un] = issued;
      }
    };
    const bool mem_first = wave < NW / 2;
    if (mem_first || !tile_full(p - 1)) memory();  // a tile that is not full is stored by every thread at once
    const bool lastp = (p == P - 1);
    char* xt = xb[u];
    float tail[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      tail[g] = 0.f;
      if (lastp && a.h_out != nullptr) {
        // sum_{j <= jstar} lambda^(jstar-j) x[16 nstar + j] (before y overwrites x)
        const int ch = cb + 4 * g + lq;
        const float2 l1 = lane_c(s_kc[kmode(g)].lam1);
        float t = 0.f;
        for (int jj = 0; jj <= jstar; ++jj) {
          const float xj = to_f32(*reinterpret_cast<const TX*>(xt + XLay<XE>::off(nstar * CHUNK + jj) + ch * XE));
          t = cfma_pair(l1.x, l1.y, t, (ln & 1) ? 0.f : xj);
        }
        tail[g] = t;
      }
    }
    // pass 2: the x operands and S of every group first, the scans (independent
    // chains, one per group) next, then per group H through LDS and
    // y = T x + U H.  On the chain's last tile the state entering chunk nstar
    // is read back from the H buffer.
    typename PT::XOp xv[NG][4];
    float S16[NG][16];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      PT::gather4(xt, cb + 4 * g, ln, lq, xv[g]);
      chunk_states<TX>(xv[g], vop[g], S16[g]);
    }
#pragma unroll
    for (int n = 0; n < 16; ++n) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const float nx = cfma_pair(mur[g], mus[g], E[g], S16[g][n]);
        S16[g][n] = E[g];  // now the state entering chunk n
        E[g] = nx;         // at the end, the state entering the next tile
      }
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
#pragma unroll
      for (int n = 0; n < 16; ++n) hs[lq * HKS + n * 16 + ln] = S16[g][n];
      wave_lds_order();
      if (lastp && a.h_out != nullptr) {
        // state at t = L-1: lambda^(jstar+1) times the state entering chunk nstar, plus the tail
        const float hn = hs[lq * HKS + nstar * 16 + ln];
        const int d = d0 + cb + 4 * g + lq, mm = ln >> 1;
        const float2 lt = lane_c(s_kc[kmode(g)].lamt);
        const float hl = cfma_pair(lt.x, lt.y, hn, tail[g]);
        if (d < a.D && mm < a.M) a.h_out[((size_t)(b * a.D + d) * a.M + mm) * 2 + (ln & 1)] = hl;
      }
      f4 acc[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const f4 hb = *reinterpret_cast<const f4*>(&hs[k * HKS + ln * 16 + 4 * lq]);
        acc[k] = PT::mma_u(uop[g][k], hb, PT::mma(top[g][k], xv[g][k], zero));
      }
      wave_lds_order();
      if (SEPY)
        put_y4_global(reinterpret_cast<float*>(a.y), acc, b, p * TILE_T + ln * CHUNK + lq * 4, d0 + cb + 4 * g,
                      a.L, a.D);
      else
        put_y4<TY>(xt, cb + 4 * g, ln, lq, acc);
    }
    if (!mem_first && tile_full(p - 1)) memory();
  }
  // the rows of the segment's last tile
  __syncthreads();
  if (!SEPY) store_tile(ubuf(S - 1), s + S - 1);

  // ---- the last work-group of a chain resets the chain's counters, the last
  // chain to finish the call's words ------------------------------------------
  if (tid == 0) {
    const uint32_t f = atomicAdd(cw + 3, 1u);
    if (f == G_ - 1) {
      st_flag(cw + 0, 0u);
      st_flag(cw + 1, 0u);
      st_flag(cw + 2, 0u);
      st_flag(cw + 3, 0u);
      if (atomicAdd(a.hdr + 2, 1u) == (uint32_t)a.nchains - 1) {
        st_flag(a.hdr + 2, 0u);
        st_flag(a.hdr + 4, 0u);
        st_flag(a.hdr + 1, ep + 1);
      }
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
                       hipStream_t st) {
  if (bwd)
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(PREP_THREADS), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(PREP_THREADS), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*, hipStream_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*, hipStream_t);

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

int fwd_stream_grid(int64_t nchains, int64_t P, int num_cus) {
  // every work-group of a chain resident at once (one per compute unit), and
  // no more of them than the chain has tiles; one per chain when there are more
  // chains than compute units (a chain is then served by one work-group alone)
  if (nchains >= num_cus) return (int)nchains;
  int64_t per = num_cus / nchains;
  if (per > P) per = P;
  if (per < 1) per = 1;
  return (int)(nchains * per);
}

template <typename TX, typename TY>
hipError_t launch_fwd_stream(const StreamArgs& a, int grid, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  launch_timed(fwd_stream_kernel<TX, TY>, dim3((unsigned)grid), dim3(StreamGeo<TX>::NT), st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_stream<float, float>(const StreamArgs&, int, hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_stream<bf16_t, bf16_t>(const StreamArgs&, int, hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_stream<bf16_t, float>(const StreamArgs&, int, hipStream_t, hipEvent_t, hipEvent_t);

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
