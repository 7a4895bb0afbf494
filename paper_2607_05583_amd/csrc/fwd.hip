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
// are 16x16x16 MFMAs whose 16 columns are the chunks of one tile (256 steps);
// all chunks share the per-channel matrices because the filter is time
// invariant.  The scan inside a tile runs one lane per (channel, mode); tiles are
// chained through per-tile end states (aggregate, then carry).
#include "common.h"
#include "tile_io.h"
#include "kernels.h"

namespace res {

// ---------------------------------------------------------------------------
// Parameter tables.  One block per (padded) channel.  Powers lambda^tau are
// evaluated in float64 from the exact integer-lag arguments tau*gamma and
// tau*omega, then rounded once to the operand type.
// ---------------------------------------------------------------------------
template <typename TA, bool BWD>
__global__ __launch_bounds__(256) void prep_kernel(const float* __restrict__ gamma,
                                                   const float* __restrict__ omega,
                                                   const float* __restrict__ amp,
                                                   const float* __restrict__ phase, int D, int M,
                                                   int MG, int last_len, TA* __restrict__ tab,
                                                   ModeScalars* __restrict__ scal,
                                                   ModeCarry* __restrict__ cc) {
  const int d = blockIdx.x;
  const int Mp = MODES_PER_GROUP * MG;
  __shared__ double2 pw[MODES_PER_GROUP * MG_MAX][CHUNK + 1];  // lambda^tau, tau = 0..16
  __shared__ double2 cm[MODES_PER_GROUP * MG_MAX];             // c
  const bool dvalid = d < D;
  for (int t = threadIdx.x; t < Mp * (CHUNK + 1); t += blockDim.x) {
    const int m = t / (CHUNK + 1), tau = t % (CHUNK + 1);
    double2 v = make_double2(0.0, 0.0);
    if (dvalid && m < M) {
      const double g = gamma[d * M + m], w = omega[d * M + m];
      const double e = exp(-g * tau);
      double s, c;
      sincos(w * tau, &s, &c);
      v = make_double2(e * c, e * s);
    }
    pw[m][tau] = v;
  }
  for (int m = threadIdx.x; m < Mp; m += blockDim.x) {
    double2 c2 = make_double2(0.0, 0.0);
    ModeScalars ms;
    ModeCarry mc;
    ms.lam = ms.mu = ms.lamT = ms.lamEll = make_float2(0.f, 0.f);
    mc.lamT = mc.lamEll = make_double2(0.0, 0.0);
    if (dvalid && m < M) {
      const double g = gamma[d * M + m], w = omega[d * M + m];
      const double a = amp[d * M + m], ph = phase[d * M + m];
      double s, c;
      sincos(ph, &s, &c);
      c2 = make_double2(a * c, a * s);
      auto powk = [&](double k) {
        double sk, ck;
        sincos(w * k, &sk, &ck);
        const double e = exp(-g * k);
        return make_double2(e * ck, e * sk);
      };
      const double2 l1 = powk(1.0), l16 = powk((double)CHUNK), lT = powk((double)TILE_T),
                    lE = powk((double)last_len);
      ms.lam = make_float2((float)l1.x, (float)l1.y);
      ms.mu = make_float2((float)l16.x, (float)l16.y);
      ms.lamT = make_float2((float)lT.x, (float)lT.y);
      ms.lamEll = make_float2((float)lE.x, (float)lE.y);
      mc.lamT = lT;
      mc.lamEll = lE;
    }
    cm[m] = c2;
    scal[(size_t)d * Mp + m] = ms;
    cc[(size_t)d * Mp + m] = mc;
  }
  __syncthreads();

  auto tap = [&](int tau) {  // K[tau] = Re sum_m c_m lambda_m^tau
    double s = 0.0;
    for (int m = 0; m < Mp; ++m) s += cm[m].x * pw[m][tau].x - cm[m].y * pw[m][tau].y;
    return s;
  };
  auto part = [](double2 z, int p) { return p ? z.y : z.x; };

  // entry (mat, i, k) of the per-channel 16x16 matrices, k = contraction index
  auto entry = [&](int mat, int i, int k) -> double {
    if (!BWD) {
      if (mat == 0) return (i >= k) ? tap(i - k) : 0.0;          // T[i][k] = K[i-k]
      const int g = (mat - 1) / 2;
      if ((mat - 1) % 2 == 0)                                     // V[comp i][k] = lambda^(15-k)
        return part(pw[g * 8 + i / 2][CHUNK - 1 - k], i & 1);
      const int m = g * 8 + k / 2;                                // U[i][comp k] = c lambda^(i+1)
      const double2 z = zmul(cm[m], pw[m][i + 1]);
      return (k & 1) ? -z.y : z.x;
    }
    if (mat == 0) return (k >= i) ? tap(k - i) : 0.0;             // Tt[j=i][k] = K[k-i]
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

  // Store in the per-lane operand layout of Path<TA>: 16 bytes per lane.
  const int nm = BWD ? bwd_mats(MG) : fwd_mats(MG);
  for (int task = threadIdx.x; task < nm * 64; task += blockDim.x) {
    const int mat = task / 64, l = task % 64, i = l % 16, q = l / 16;
    uint4 out;
    if (sizeof(TA) == 4) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (float)entry(mat, i, 4 * q + r);
      out = *reinterpret_cast<const uint4*>(v);
    } else {
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
// Forward tile kernel.
//   MODE_STATE: chunk states -> scan -> tile aggregate (end state of the tile from
//               its own drives, zero state entering); the last tile of a row
//               writes the state at t = L-1 instead.  Writes agg[b][p][d][m].
//   MODE_APPLY: reads the state entering the tile (carry[b][p][d][m]) and writes y.
// ---------------------------------------------------------------------------
template <typename TX, typename TY, int MG, int MODE>
__global__ __launch_bounds__(NTHREADS) void fwd_tile_kernel(FwdArgs a) {
  typedef Path<TX> PT;
  constexpr int DW = tile_channels<TX>();
  constexpr int CPW = DW / NWAVES;  // channels per wave
  constexpr int NCG = CPW / 8;      // scan groups of 8 channels per wave
  typedef TileGeom<TX, DW> GX;
  constexpr int XP = GX::PITCH;
  constexpr int NSTR = 16 * MG;         // floats per chunk in the scan buffer
  constexpr int KSTR = 16 * NSTR + 16;  // floats per channel in the scan buffer
  constexpr int WSB = 8 * KSTR;         // floats per wave
  constexpr bool SEPY = !__is_same(TX, TY);
  typedef TileGeom<float, DW> GY;

  // The fp32 output tile of the bf16 -> f32 variant reuses the scan buffer, which
  // is free once the correction products are done.
  constexpr int SBUF = (SEPY && DW * GY::PITCH > NWAVES * WSB) ? DW * GY::PITCH : NWAVES * WSB;
  __shared__ __align__(16) TX xt[DW * XP];
  __shared__ __align__(16) float sbuf[SBUF];
  float* ytf = sbuf;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, lq = lane >> 4;  // MFMA lane coordinates
  const int sk = lane >> 3, sj = lane & 7;   // scan lane: channel in group, mode in group

  const int64_t tile = blockIdx.x;
  const int nb = (int)(tile % a.NB);
  const int64_t rest = tile / a.NB;
  const int64_t b = rest % a.B;
  const int64_t p = rest / a.B;
  const int64_t t0 = p * TILE_T;
  const int d0 = nb * DW;
  const bool last = (p == a.P - 1);

  load_tile<TX, DW>(reinterpret_cast<const TX*>(a.x), xt, b, t0, d0, a.L, a.D, tid);
  __syncthreads();

  const char* tab = reinterpret_cast<const char*>(a.tab);
  constexpr int NM = 1 + 2 * MG;
  float* sb = sbuf + wave * WSB;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};

  f4 yacc[CPW];
  float2 hx[NCG][MG][NCHUNK];
  float2 aggv[NCG][MG];

#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ch = wave * CPW + cg * 8 + k;
      const char* tp = tab + (size_t)(d0 + ch) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
      const typename PT::XOp xv = PT::load_x(&xt[ch * XP + PT::x_off(li, lq)]);
      if (MODE == MODE_APPLY) yacc[cg * 8 + k] = PT::mma(PT::load_a(tp), xv, zero);
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const f4 s = PT::mma(PT::load_a(tp + (1 + 2 * g) * TAB_MAT_BYTES), xv, zero);
        *reinterpret_cast<f4*>(&sb[k * KSTR + li * NSTR + g * 16 + lq * 4]) = s;
      }
    }
    __syncthreads();
    {
      const int ch = wave * CPW + cg * 8 + sk;
      const int dch = d0 + ch;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int m = g * 8 + sj;
        const float2 mu = a.scal[(size_t)dch * a.Mp + m].mu;
        float2 run = make_float2(0.f, 0.f);
#pragma unroll
        for (int n = 0; n < NCHUNK; ++n) {
          hx[cg][g][n] = run;
          const float2 s = *reinterpret_cast<const float2*>(&sb[sk * KSTR + n * NSTR + g * 16 + 2 * sj]);
          run = cfma(mu, run, s);
        }
        aggv[cg][g] = run;
      }
    }
    __syncthreads();
  }

  if (MODE == MODE_STATE) {
    const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg) {
      const int ch = wave * CPW + cg * 8 + sk;
      const int dch = d0 + ch;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int m = g * 8 + sj;
        float2 v = aggv[cg][g];
        if (last) {
          // state at t = L-1: enter chunk nstar, then step through its valid drives
          float2 h = hx[cg][g][0];
#pragma unroll
          for (int n = 1; n < NCHUNK; ++n)
            if (n == nstar) h = hx[cg][g][n];
          const float2 lam = a.scal[(size_t)dch * a.Mp + m].lam;
          for (int j = 0; j <= jstar; ++j) {
            const float xvv = to_f32(xt[ch * XP + nstar * CHUNK + j]);
            h = cfma(lam, h, make_float2(xvv, 0.f));
          }
          v = h;
        }
        a.agg[((size_t)(b * a.P + p) * a.Dp + dch) * a.Mp + m] = v;
      }
    }
    return;
  }

  // MODE_APPLY: add the carried state, then the correction product.
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    {
      const int ch = wave * CPW + cg * 8 + sk;
      const int dch = d0 + ch;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const int m = g * 8 + sj;
        const float2 mu = a.scal[(size_t)dch * a.Mp + m].mu;
        float2 w = a.carry[((size_t)(b * a.P + p) * a.Dp + dch) * a.Mp + m];
#pragma unroll
        for (int n = 0; n < NCHUNK; ++n) {
          const float2 h = make_float2(hx[cg][g][n].x + w.x, hx[cg][g][n].y + w.y);
          *reinterpret_cast<float2*>(&sb[sk * KSTR + n * NSTR + g * 16 + 2 * sj]) = h;
          w = cmul(mu, w);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ch = wave * CPW + cg * 8 + k;
      const char* tp = tab + (size_t)(d0 + ch) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const float* hv = &sb[k * KSTR + li * NSTR + g * 16 + PT::h_off(lq)];
        yacc[cg * 8 + k] = PT::mma_state(PT::load_a(tp + (2 + 2 * g) * TAB_MAT_BYTES), hv, yacc[cg * 8 + k]);
      }
    }
    __syncthreads();
  }

  // y -> LDS (in place of x, or a separate fp32 tile) -> HBM
#pragma unroll
  for (int c = 0; c < CPW; ++c) {
    const int ch = wave * CPW + c;
    if (SEPY) {
      *reinterpret_cast<f4*>(&ytf[ch * GY::PITCH + li * CHUNK + lq * 4]) = yacc[c];
    } else {
      TY v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = from_f32<TY>(yacc[c][r]);
      TY* dst = reinterpret_cast<TY*>(xt) + ch * XP + li * CHUNK + lq * 4;
      if (sizeof(TY) == 2) {
        *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(v);
      } else {
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(v);
      }
    }
  }
  __syncthreads();
  if (SEPY) {
    store_tile<float, DW>(reinterpret_cast<float*>(a.y), ytf, b, t0, d0, a.L, a.D, tid);
  } else {
    store_tile<TY, DW>(reinterpret_cast<TY*>(a.y), reinterpret_cast<const TY*>(xt), b, t0, d0, a.L,
                       a.D, tid);
  }
}

// ---------------------------------------------------------------------------
// Cross-tile carry: for each (b, d, m), in float64,
//   carry[p] = state entering tile p (carry[0] = h0),
//   carry[p+1] = lambda^TILE_T carry[p] + agg[p],
//   final state h_{L-1} = lambda^last_len carry[P-1] + agg[P-1].
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void carry_fwd_kernel(const float2* __restrict__ agg,
                                                        float2* __restrict__ carry,
                                                        const float* __restrict__ h0,
                                                        float* __restrict__ hout,
                                                        const ModeCarry* __restrict__ cc, int B,
                                                        int64_t P, int D, int M, int Dp, int Mp) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * Dp * Mp) return;
  const int m = (int)(idx % Mp);
  const int d = (int)((idx / Mp) % Dp);
  const int64_t b = idx / ((int64_t)Mp * Dp);
  const bool valid = d < D && m < M;
  const size_t sidx = ((size_t)(b * D + d) * M + m) * 2;
  double2 h = make_double2(0.0, 0.0);
  if (h0 != nullptr && valid) h = make_double2(h0[sidx], h0[sidx + 1]);
  const ModeCarry c = cc[(size_t)d * Mp + m];
  constexpr int BATCH = 16;
  for (int64_t p0 = 0; p0 < P; p0 += BATCH) {
    float2 ag[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int64_t p = p0 + j;
      ag[j] = (p < P) ? agg[((size_t)(b * P + p) * Dp + d) * Mp + m] : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int64_t p = p0 + j;
      if (p < P) {
        if (carry != nullptr)
          carry[((size_t)(b * P + p) * Dp + d) * Mp + m] = make_float2((float)h.x, (float)h.y);
        const double2 prop = (p < P - 1) ? c.lamT : c.lamEll;
        h = zfma(prop, h, make_double2((double)ag[j].x, (double)ag[j].y));
      }
    }
  }
  if (hout != nullptr && valid) {
    hout[sidx] = (float)h.x;
    hout[sidx + 1] = (float)h.y;
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
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       hipStream_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*,
                                        hipStream_t);

template <typename TX, typename TY>
hipError_t launch_fwd_tile(const Geometry& g, int mode, const FwdArgs& a, hipStream_t st,
                           hipEvent_t ev0, hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1) {
    if (mode == MODE_STATE)
      launch_timed(fwd_tile_kernel<TX, TY, 1, MODE_STATE>, grid, block, st, ev0, ev1, a);
    else
      launch_timed(fwd_tile_kernel<TX, TY, 1, MODE_APPLY>, grid, block, st, ev0, ev1, a);
  } else {
    if (mode == MODE_STATE)
      launch_timed(fwd_tile_kernel<TX, TY, 2, MODE_STATE>, grid, block, st, ev0, ev1, a);
    else
      launch_timed(fwd_tile_kernel<TX, TY, 2, MODE_APPLY>, grid, block, st, ev0, ev1, a);
  }
  return hipGetLastError();
}
template hipError_t launch_fwd_tile<float, float>(const Geometry&, int, const FwdArgs&,
                                                   hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_tile<bf16_t, bf16_t>(const Geometry&, int, const FwdArgs&,
                                                   hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_tile<bf16_t, float>(const Geometry&, int, const FwdArgs&,
                                                   hipStream_t, hipEvent_t, hipEvent_t);

hipError_t launch_carry_fwd(const Geometry& g, const float2* agg, float2* carry, const float* h0,
                            float* hout, const ModeCarry* cc, hipStream_t st) {
  const int64_t n = g.B * (int64_t)g.Dp * g.Mp;
  hipLaunchKernelGGL(carry_fwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, agg,
                     carry, h0, hout, cc, (int)g.B, g.P, (int)g.D, (int)g.M, g.Dp, g.Mp);
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace res
