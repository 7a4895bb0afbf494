// Backward of the resonant mixing operator for gfx950.
//
// With y_t = Re sum_m c_m h_{m,t}, h_t = lambda h_{t-1} + x_t (Sec. 3.1 kernel,
// Sec. 3.3 recurrence) and upstream gradient dy, define the adjoint states
//   q_s   = sum_{t>=s} lambda^(t-s) dy_t            (reverse recurrence)
//   rho_s = sum_{t>=s} (t-s) lambda^(t-s) dy_t       (lag-weighted)
// Then dx_s = Re sum_m c_m q_s, and with W = sum_s x_s q_s, R = sum_s x_s rho_s:
//   damp = Re(e^{i phi} W), dphase = -Im(c W), dgamma = -Re(c R), domega = -Im(c R)
// (plus the h0 terms, see bwd_reduce_kernel).
//
// Chunked form (chunk n = steps 16n..16n+15, Qin[n], rin[n] = (q, rho) at 16(n+1)):
//   dx[16n+j]  = sum_{i>=j} K[i-j] dy[16n+i] + Re sum_m c lambda^(16-j) Qin[n]  Tt, Ub
//   Eq[n] = sum_i lambda^i dy[16n+i],  Er[n] = sum_i i lambda^i dy[16n+i]          Eq, Er
//   Qin[n-1] = Eq[n] + mu Qin[n],  rin[n-1] = Er[n] + mu (16 Qin[n] + rin[n])     reverse scan
//   W = sum_n Xs[n] Qin[n] + sum_tau lambda^tau G[tau]
//   R = sum_n (Xw[n] Qin[n] + Xs[n] rin[n]) + sum_tau tau lambda^tau G[tau]
//   Xs[n] = sum_j lambda^(16-j) x[16n+j],  Xw[n] = sum_j (16-j) lambda^(16-j) x[16n+j]
//   G[tau] = sum_n sum_j dy[16n+j+tau] x[16n+j]   (diagonal sums of P = DY X^T)
// Every product is a 16x16x16 MFMA per channel over the 16 chunks of a tile; the
// sums over chunks of Xs Qin etc. are MFMAs contracting over the chunk index.
#include "common.h"
#include "kernels.h"
#include "tile_io.h"

namespace res {

// Four activations at steps 16(4q + r) + i, r = 0..3, of one LDS tile row: the
// operand that contracts over the tile's chunks.
__device__ __forceinline__ s4 chunk_gather(const bf16_t* row, int i, int q) {
  s4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = (short)row[CHUNK * (4 * q + r) + i];
  return v;
}
__device__ __forceinline__ f4 chunk_gather(const float* row, int i, int q) {
  f4 v;
#pragma unroll
  for (int r = 0; r < 4; ++r) v[r] = row[CHUNK * (4 * q + r) + i];
  return v;
}

// Layout of the per-tile partial sums: [G(16) | per mode (W re, W im, R re, R im)].
__host__ __device__ inline int part_stride(int Mp) { return 16 + 4 * Mp; }

// A block of BW_WAVES waves takes one tile; each wave owns CPW channels and
// works through them in groups of GS (the scan uses GS x 8 lanes, one per
// (channel, mode)).  Eight waves of 8 channels hold the same LDS as four waves
// of 16 would, with twice the waves to hide latency.
constexpr int BW_WAVES = 8;
constexpr int BW_THREADS = 64 * BW_WAVES;

template <typename TX, int MG, int MODE>
__global__ __launch_bounds__(BW_THREADS) void bwd_tile_kernel(BwdArgs a) {
  typedef Path<TX> PT;
  typedef typename PT::XOp XOp;
  constexpr int DW = tile_channels<TX>();
  constexpr int GS = 4;                  // channels per group
  constexpr int CPW = DW / BW_WAVES;
  constexpr int NCG = CPW / GS;
  static_assert(CPW % GS == 0, "a wave's channels split into whole groups");
  typedef TileGeom<TX, DW> GX;
  constexpr int XP = GX::PITCH;
  // Mode groups are processed one after another; the scan buffer holds one group.
  constexpr int NSTR = 36;               // floats per chunk: 16 Q comps | 16 rho comps | 4 pad (banks)
  constexpr int KSTR = 16 * NSTR + 16;   // floats per channel
  constexpr int WSB = GS * KSTR;         // floats per wave
  constexpr int NM = 1 + 5 * MG;
  constexpr int PP = 17;                 // row pitch of the P dump (odd: rows on distinct banks)
  constexpr int PDW = 16 * PP;           // DW pairs after P
  constexpr int PST = PDW + 64 + 4;      // dump per channel: P | DW pairs | DR pairs | pad (banks)

  __shared__ __align__(16) TX dyt[DW * XP];
  __shared__ __align__(16) TX xt[MODE == MODE_APPLY ? DW * XP : 8];
  __shared__ __align__(16) float sbuf[BW_WAVES * WSB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, lq = lane >> 4;
  const int sk = lane >> 3, sj = lane & 7;

  const int64_t tile = blockIdx.x;
  const int nb = (int)(tile % a.NB);
  const int64_t rest = tile / a.NB;
  const int64_t b = rest % a.B;
  const int64_t p = rest / a.B;
  const int64_t t0 = p * TILE_T;
  const int d0 = nb * DW;

  if (tid < NTHREADS) {  // the tile movers are written for NWAVES waves
    load_tile_any<TX, DW>(reinterpret_cast<const TX*>(a.dy), dyt, b, t0, d0, a.L, a.D, tid);
    if (MODE == MODE_APPLY)
      load_tile_any<TX, DW>(reinterpret_cast<const TX*>(a.x), xt, b, t0, d0, a.L, a.D, tid);
  }
  __syncthreads();

  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* sb = sbuf + wave * WSB;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  const size_t tm = (size_t)(b * a.P + p) * a.Dp;  // tile row in [B][P][Dp]
  static_assert(GS * PST <= WSB, "reduction dump must fit the scan buffer");

#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    f4 dxacc[GS];
    f4 pacc[GS];
    if (MODE == MODE_APPLY) {
#pragma unroll
      for (int k = 0; k < GS; ++k) {
        const int ch = wave * CPW + cg * GS + k;
        const char* tp = tab + (size_t)(d0 + ch) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
        const XOp dyv = PT::load_x(&dyt[ch * XP + PT::x_off(li, lq)]);
        dxacc[k] = PT::mma(PT::load_a(tp), dyv, zero);
        // P = DY X^T, contracting over the tile's chunks (exact products)
        pacc[k] = mma_k16_act(chunk_gather(&dyt[ch * XP], li, lq), chunk_gather(&xt[ch * XP], li, lq),
                              zero);
      }
    }
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      // ---- chunk sums of dy: Eq, Er -------------------------------------------
#pragma unroll
      for (int k = 0; k < GS; ++k) {
        const int ch = wave * CPW + cg * GS + k;
        const char* tp = tab + (size_t)(d0 + ch) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
        const XOp dyv = PT::load_x(&dyt[ch * XP + PT::x_off(li, lq)]);
        const f4 eq = PT::mma(PT::load_a(tp + (1 + 5 * g) * TAB_MAT_BYTES), dyv, zero);
        const f4 er = PT::mma(PT::load_a(tp + (2 + 5 * g) * TAB_MAT_BYTES), dyv, zero);
        *reinterpret_cast<f4*>(&sb[k * KSTR + li * NSTR + lq * 4]) = eq;
        *reinterpret_cast<f4*>(&sb[k * KSTR + li * NSTR + 16 + lq * 4]) = er;
      }
      __syncthreads();
      // ---- reverse scan over the tile's chunks, one lane per (channel, mode) ---
      if (sk < GS) {
        const int ch = wave * CPW + cg * GS + sk;
        const int dch = d0 + ch;
        const int m = g * 8 + sj;
        const float2 mu = a.scal[(size_t)dch * a.Mp + m].mu;
        float2 Q = make_float2(0.f, 0.f), Rr = Q;
        float2 wQ = Q, wR = Q;
        if (MODE == MODE_APPLY) {
          const float4 c = a.carry[(tm + dch) * a.Mp + m];
          wQ = make_float2(c.x, c.y);
          wR = make_float2(c.z, c.w);
        }
        float* eqp = &sb[sk * KSTR + 2 * sj];
        float* erp = eqp + 16;
#pragma unroll
        for (int n = NCHUNK - 1; n >= 0; --n) {
          const float2 eq = *reinterpret_cast<const float2*>(eqp + n * NSTR);
          const float2 er = *reinterpret_cast<const float2*>(erp + n * NSTR);
          if (MODE == MODE_APPLY) {
            // (q, rho) entering chunk n from the right: local part + propagated carry
            *reinterpret_cast<float2*>(eqp + n * NSTR) = make_float2(Q.x + wQ.x, Q.y + wQ.y);
            *reinterpret_cast<float2*>(erp + n * NSTR) = make_float2(Rr.x + wR.x, Rr.y + wR.y);
            const float2 nwQ = cmul(mu, wQ);
            wR = cmul(mu, make_float2(fmaf(16.f, wQ.x, wR.x), fmaf(16.f, wQ.y, wR.y)));
            wQ = nwQ;
          }
          const float2 nQ = cfma(mu, Q, eq);
          Rr = cfma(mu, make_float2(fmaf(16.f, Q.x, Rr.x), fmaf(16.f, Q.y, Rr.y)), er);
          Q = nQ;
        }
        if (MODE == MODE_STATE) a.agg[(tm + dch) * a.Mp + m] = make_float4(Q.x, Q.y, Rr.x, Rr.y);
      }
      __syncthreads();
      if (MODE == MODE_STATE) continue;

      // ---- dx correction, chunk sums of x, cross products over chunks ---------
      f4 dwacc[GS], dracc[GS];
#pragma unroll
      for (int k = 0; k < GS; ++k) {
        const int ch = wave * CPW + cg * GS + k;
        const char* tp = tab + (size_t)(d0 + ch) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
        const XOp xv = PT::load_x(&xt[ch * XP + PT::x_off(li, lq)]);
        const float* srow = &sb[k * KSTR];
        // dx += Ub Qin (float32 product of the carried states)
        dxacc[k] = mma_f32(load_f4(tp + (5 + 5 * g) * TAB_MAT_BYTES),
                           load_f4(&srow[li * NSTR + lq * 4]), dxacc[k]);
        // Xs^T, Xw^T: rows = chunks, columns = components (the table is the B operand)
        const f4 xs = PT::mma(xv, PT::load_a(tp + (3 + 5 * g) * TAB_MAT_BYTES), zero);
        const f4 xw = PT::mma(xv, PT::load_a(tp + (4 + 5 * g) * TAB_MAT_BYTES), zero);
        // Qin^T, rin^T contracting over chunks: lane (comp, q) holds chunks 4q..4q+3
        f4 qt, rt;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          qt[r] = srow[(4 * lq + r) * NSTR + li];
          rt[r] = srow[(4 * lq + r) * NSTR + 16 + li];
        }
        dwacc[k] = mma_f32(xs, qt, zero);
        dracc[k] = mma_f32(xs, rt, mma_f32(xw, qt, zero));
      }
      __syncthreads();
      // ---- dump P (first group) and the 2x2 diagonal blocks, then reduce -------
#pragma unroll
      for (int k = 0; k < GS; ++k) {
        float* dst = &sb[k * PST];
        if (g == 0) {
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[(4 * lq + r) * PP + li] = pacc[k][r];
        }
        // lane (col li, q) holds rows 4q..4q+3; the 2x2 diagonal blocks are in lanes li/4 == q
        if ((li >> 2) == lq) {
          const int r0 = li & 2;  // rows li&~1 and li|1
          dst[PDW + li * 2 + 0] = dwacc[k][r0];
          dst[PDW + li * 2 + 1] = dwacc[k][r0 + 1];
          dst[PDW + 32 + li * 2 + 0] = dracc[k][r0];
          dst[PDW + 32 + li * 2 + 1] = dracc[k][r0 + 1];
        }
      }
      __syncthreads();
      if (sk < GS) {
        // lane (sk, sj): channel sk of the group; G[sj], G[sj + 8]; mode g*8 + sj
        const int ch = wave * CPW + cg * GS + sk;
        const int dch = d0 + ch;
        const float* src = &sb[sk * PST];
        float* out = a.part + (tm + dch) * part_stride(a.Mp);
        if (g == 0) {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int tau = sj + 8 * h;
            float s = 0.f;
            for (int j = 0; j + tau < 16; ++j) s += src[(j + tau) * PP + j];
            out[tau] = s;
          }
        }
        // column c holds (D[c&~1][c], D[c|1][c]) at [2c], [2c+1]
        const float* dwp = &src[PDW];
        const float* drp = dwp + 32;
        const int c0 = 2 * sj, c1 = 2 * sj + 1;
        const float w_rr = dwp[2 * c0], w_ir = dwp[2 * c0 + 1], w_ri = dwp[2 * c1], w_ii = dwp[2 * c1 + 1];
        const float r_rr = drp[2 * c0], r_ir = drp[2 * c0 + 1], r_ri = drp[2 * c1], r_ii = drp[2 * c1 + 1];
        float4 v;
        v.x = w_rr - w_ii;
        v.y = w_ri + w_ir;
        v.z = r_rr - r_ii;
        v.w = r_ri + r_ir;
        *reinterpret_cast<float4*>(&out[16 + 4 * (g * 8 + sj)]) = v;
      }
      __syncthreads();
    }
    if (MODE == MODE_APPLY) {
      // dx -> LDS in place of dy (each wave owns its channels' rows)
#pragma unroll
      for (int k = 0; k < GS; ++k) {
        const int ch = wave * CPW + cg * GS + k;
        TX v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = from_f32<TX>(dxacc[k][r]);
        TX* dst = &dyt[ch * XP + li * CHUNK + lq * 4];
        if (sizeof(TX) == 2)
          *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(v);
        else
          *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(v);
      }
    }
  }
  if (MODE == MODE_APPLY) {
    __syncthreads();
    if (tid < NTHREADS) store_tile_any<TX, DW>(reinterpret_cast<TX*>(a.dx), dyt, b, t0, d0, a.L, a.D, tid);
  }
}

// ---------------------------------------------------------------------------
// Cross-tile carry, right to left, in float64.  With Incl(p) the (q, rho) pair at
// the left edge of tile p from all drives at or after it:
//   carry[p]  = Incl(p+1)  (state entering tile p from the right; 0 for the last)
//   Incl(p)   = agg[p] + (Lambda Incl_q, Lambda (TILE_T Incl_q + Incl_rho))(p+1)
//   q0[b,d,m] = Incl(0)   ((q, rho) at t = 0)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void carry_bwd_kernel(const float4* __restrict__ agg,
                                                        float4* __restrict__ carry,
                                                        float4* __restrict__ q0,
                                                        const ModeCarry* __restrict__ cc, int B,
                                                        int64_t P, int Dp, int Mp) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * Dp * Mp) return;
  const int m = (int)(idx % Mp);
  const int d = (int)((idx / Mp) % Dp);
  const int64_t b = idx / ((int64_t)Mp * Dp);
  const double2 lT = cc[(size_t)d * Mp + m].lamT;
  double2 Q = make_double2(0.0, 0.0), Rr = Q;
  constexpr int BATCH = 16;
  for (int64_t p1 = P - 1; p1 >= 0; p1 -= BATCH) {
    float4 ag[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      // past the first tile the index is clamped (the value is not used), so
      // the loads are unconditional and all of them are in flight at once
      const int64_t p = p1 - j >= 0 ? p1 - j : 0;
      ag[j] = agg[((size_t)(b * P + p) * Dp + d) * Mp + m];
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      const int64_t p = p1 - j;
      if (p >= 0) {
        carry[((size_t)(b * P + p) * Dp + d) * Mp + m] =
            make_float4((float)Q.x, (float)Q.y, (float)Rr.x, (float)Rr.y);
        // propagate over tile p (TILE_T steps), then add its own aggregate
        const double2 tq = make_double2(fma((double)TILE_T, Q.x, Rr.x), fma((double)TILE_T, Q.y, Rr.y));
        Rr = zfma(lT, tq, make_double2(ag[j].z, ag[j].w));
        Q = zfma(lT, Q, make_double2(ag[j].x, ag[j].y));
      }
    }
  }
  q0[((size_t)b * Dp + d) * Mp + m] = make_float4((float)Q.x, (float)Q.y, (float)Rr.x, (float)Rr.y);
}

// ---------------------------------------------------------------------------
// Fixed-order reduction of the per-tile partials (float64), one block per channel d:
//   W = sum_tiles W_inter + sum_tau lambda^tau G[tau] + sum_b lambda q0 h0
//   R = sum_tiles R_inter + sum_tau tau lambda^tau G[tau] + sum_b lambda (q0 + rho0) h0
//   damp = Re(e^{i phi} W), dphase = -Im(c W), dgamma = -Re(c R), domega = -Im(c R)
//   dh0[b,d,m] = (Re(c lambda q0), -Im(c lambda q0))
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_reduce_kernel(
    const float* __restrict__ part, const float4* __restrict__ q0, const float* __restrict__ gamma,
    const float* __restrict__ omega, const float* __restrict__ amp, const float* __restrict__ phase,
    const float* __restrict__ h0, float* __restrict__ dgamma, float* __restrict__ domega,
    float* __restrict__ damp, float* __restrict__ dphase, float* __restrict__ dh0, int B,
    int64_t P, int D, int M, int Dp, int Mp) {
  // One block per channel d.  The ps columns of the per-tile partial rows of d
  // are summed over the B P tiles in float64: thread (row group rg, column col)
  // takes tiles rg, rg + NRG, ... into eight interleaved accumulators (eight
  // loads in flight), then the row groups are added in order.  The order is
  // fixed, so the result is bitwise reproducible.
  const int d = blockIdx.x;
  const int ps = part_stride(Mp);
  const int nrg = blockDim.x / ps;
  const int64_t nbp = (int64_t)B * P;
  __shared__ double s_acc[256];
  __shared__ double s_col[16 + 4 * MODES_PER_GROUP * MG_MAX];
  {
    const int col = threadIdx.x % ps, rg = threadIdx.x / ps;
    double acc = 0.0;
    if (rg < nrg) {
      double ac[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
      int64_t bp = rg;
      for (; bp + 7 * nrg < nbp; bp += 8 * nrg) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = part[((size_t)(bp + u * nrg) * Dp + d) * ps + col];
#pragma unroll
        for (int u = 0; u < 8; ++u) ac[u] += v[u];
      }
      for (; bp < nbp; bp += nrg) ac[0] += part[((size_t)bp * Dp + d) * ps + col];
      acc = ((ac[0] + ac[1]) + (ac[2] + ac[3])) + ((ac[4] + ac[5]) + (ac[6] + ac[7]));
    }
    s_acc[threadIdx.x] = acc;
  }
  __syncthreads();
  for (int col = threadIdx.x; col < ps; col += blockDim.x) {
    double t = 0.0;
    for (int rg = 0; rg < nrg; ++rg) t += s_acc[rg * ps + col];
    s_col[col] = t;
  }
  __syncthreads();
  const int m = threadIdx.x;
  if (m >= M) return;
  const int idx = d * M + m;
  double G[16];
#pragma unroll
  for (int t = 0; t < 16; ++t) G[t] = s_col[t];
  double Wr = s_col[16 + 4 * m], Wi = s_col[16 + 4 * m + 1], Rr = s_col[16 + 4 * m + 2],
         Ri = s_col[16 + 4 * m + 3];
  const double g = gamma[idx], w = omega[idx], a = amp[idx], ph = phase[idx];
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    double s, c;
    sincos(w * t, &s, &c);
    const double e = exp(-g * t);
    Wr += e * c * G[t];
    Wi += e * s * G[t];
    Rr += t * e * c * G[t];
    Ri += t * e * s * G[t];
  }
  double sp, cp, sw, cw;
  sincos(ph, &sp, &cp);
  sincos(w, &sw, &cw);
  const double el = exp(-g);
  const double2 lam = make_double2(el * cw, el * sw);
  const double2 cc = make_double2(a * cp, a * sp);
  const double2 cl = zmul(cc, lam);
  for (int b = 0; b < B; ++b) {
    const float4 qq = q0[((size_t)b * Dp + d) * Mp + m];
    const double2 qz = make_double2(qq.x, qq.y), rz = make_double2(qq.z, qq.w);
    if (h0 != nullptr) {
      const size_t s = ((size_t)(b * D + d) * M + m) * 2;
      const double2 hz = make_double2(h0[s], h0[s + 1]);
      const double2 lw = zmul(zmul(lam, qz), hz);
      const double2 lr = zmul(zmul(lam, make_double2(qz.x + rz.x, qz.y + rz.y)), hz);
      Wr += lw.x;
      Wi += lw.y;
      Rr += lr.x;
      Ri += lr.y;
    }
    if (dh0 != nullptr) {
      const double2 z = zmul(cl, qz);
      const size_t s = ((size_t)(b * D + d) * M + m) * 2;
      dh0[s] = (float)z.x;
      dh0[s + 1] = (float)(-z.y);
    }
  }
  const double2 cW = zmul(cc, make_double2(Wr, Wi));
  const double2 cR = zmul(cc, make_double2(Rr, Ri));
  damp[idx] = (float)(cp * Wr - sp * Wi);  // Re(e^{i phi} W)
  dphase[idx] = (float)(-cW.y);
  dgamma[idx] = (float)(-cR.x);
  domega[idx] = (float)(-cR.y);
}

// ---------------------------------------------------------------------------
template <typename TX>
hipError_t launch_bwd_tile(const Geometry& g, int mode, const BwdArgs& a, hipStream_t st,
                           hipEvent_t ev0, hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(BW_THREADS);
  if (g.MG == 1) {
    if (mode == MODE_STATE)
      launch_timed(bwd_tile_kernel<TX, 1, MODE_STATE>, grid, block, st, ev0, ev1, a);
    else
      launch_timed(bwd_tile_kernel<TX, 1, MODE_APPLY>, grid, block, st, ev0, ev1, a);
  } else {
    if (mode == MODE_STATE)
      launch_timed(bwd_tile_kernel<TX, 2, MODE_STATE>, grid, block, st, ev0, ev1, a);
    else
      launch_timed(bwd_tile_kernel<TX, 2, MODE_APPLY>, grid, block, st, ev0, ev1, a);
  }
  return hipGetLastError();
}
template hipError_t launch_bwd_tile<float>(const Geometry&, int, const BwdArgs&, hipStream_t,
                                           hipEvent_t, hipEvent_t);
template hipError_t launch_bwd_tile<bf16_t>(const Geometry&, int, const BwdArgs&, hipStream_t,
                                            hipEvent_t, hipEvent_t);

hipError_t launch_carry_bwd(const Geometry& g, const float4* agg, float4* carry, float4* q0,
                            const ModeCarry* cc, hipStream_t st) {
  const int64_t n = g.B * (int64_t)g.Dp * g.Mp;
  hipLaunchKernelGGL(carry_bwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, agg,
                     carry, q0, cc, (int)g.B, g.P, g.Dp, g.Mp);
  return hipGetLastError();
}

hipError_t launch_bwd_reduce(const Geometry& g, const float* part, const float4* q0,
                             const float* gamma, const float* omega, const float* amp,
                             const float* phase, const float* h0, float* dgamma, float* domega,
                             float* damp, float* dphase, float* dh0, hipStream_t st) {
  hipLaunchKernelGGL(bwd_reduce_kernel, dim3((unsigned)g.D), dim3(256), 0, st, part,
                     q0, gamma, omega, amp, phase, h0, dgamma, domega, damp, dphase, dh0,
                     (int)g.B, g.P, (int)g.D, (int)g.M, g.Dp, g.Mp);
  return hipGetLastError();
}

}  // namespace res
