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
// Inside a tile the chunk scan runs one lane per (channel, mode).  Across tiles
// the state is chained in a single pass (decoupled look-back): each tile
// publishes the end state of its own drives, then the state entering it,
// computed from its predecessors' published states.
#include "common.h"
#include "kernels.h"
#include "tile_io.h"

namespace res {

// ---------------------------------------------------------------------------
// Parameter tables.  One block per (padded) channel.  lambda and c come from one
// float64 exp/sincos each; lambda^tau (tau <= 16) by float64 products,
// lambda^256 by squaring, lambda^last_len by binary powering (relative error
// ~1e-14, far below float32 resolution).  Entries are rounded once to the
// operand type.  The grid also clears the flags of the chained scan.
// ---------------------------------------------------------------------------
template <typename TA, bool BWD>
__global__ __launch_bounds__(256) void prep_kernel(const float* __restrict__ gamma,
                                                   const float* __restrict__ omega,
                                                   const float* __restrict__ amp,
                                                   const float* __restrict__ phase, int D, int M,
                                                   int MG, int last_len, TA* __restrict__ tab,
                                                   ModeScalars* __restrict__ scal,
                                                   ModeCarry* __restrict__ cc,
                                                   uint32_t* __restrict__ flags, int64_t nflags) {
  const int d = blockIdx.x;
  const int Mp = MODES_PER_GROUP * MG;
  __shared__ double2 pw[MODES_PER_GROUP * MG_MAX][CHUNK + 1];  // lambda^tau, tau = 0..16
  __shared__ double2 cm[MODES_PER_GROUP * MG_MAX];             // c
  __shared__ double ev[MODES_PER_GROUP * MG_MAX][5];           // e^-g, cos w, sin w, cos p, sin p
  __shared__ double taps[CHUNK + 1];

  if (flags != nullptr) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nflags;
         i += (int64_t)gridDim.x * blockDim.x)
      flags[i] = FLAG_NONE;
  }

  const bool dvalid = d < D;
  // one transcendental per thread: (m, which) with which = exp | sincos(omega) | sincos(phi)
  for (int t = threadIdx.x; t < Mp * 3; t += blockDim.x) {
    const int m = t / 3, which = t % 3;
    if (dvalid && m < M) {
      if (which == 0) {
        ev[m][0] = exp(-(double)gamma[d * M + m]);
      } else {
        double s, c;
        sincos(which == 1 ? (double)omega[d * M + m] : (double)phase[d * M + m], &s, &c);
        ev[m][2 * which - 1] = c;
        ev[m][2 * which] = s;
      }
    } else {
      if (which == 0) {
        ev[m][0] = 0.0;
      } else {
        ev[m][2 * which - 1] = 0.0;
        ev[m][2 * which] = 0.0;
      }
    }
  }
  __syncthreads();
  for (int m = threadIdx.x; m < Mp; m += blockDim.x) {
    const bool valid = dvalid && m < M;
    const double a = valid ? (double)amp[d * M + m] : 0.0;
    const double2 lam = make_double2(ev[m][0] * ev[m][1], ev[m][0] * ev[m][2]);
    cm[m] = make_double2(a * ev[m][3], a * ev[m][4]);
    double2 pk = make_double2(valid ? 1.0 : 0.0, 0.0);
    for (int tau = 0; tau <= CHUNK; ++tau) {
      pw[m][tau] = pk;
      pk = zmul(pk, lam);
    }
    double2 lT = pw[m][CHUNK];                      // lambda^16 -> lambda^256
    for (int s = 0; s < 4; ++s) lT = zmul(lT, lT);
    double2 lE = make_double2(valid ? 1.0 : 0.0, 0.0), base = lam;  // lambda^last_len
    for (int e = last_len; e > 0; e >>= 1) {
      if (e & 1) lE = zmul(lE, base);
      base = zmul(base, base);
    }
    ModeScalars ms;
    ms.lam = make_float2((float)lam.x, (float)lam.y);
    ms.mu = make_float2((float)pw[m][CHUNK].x, (float)pw[m][CHUNK].y);
    ms.lamT = make_float2((float)lT.x, (float)lT.y);
    ms.lamEll = make_float2((float)lE.x, (float)lE.y);
    scal[(size_t)d * Mp + m] = ms;
    ModeCarry mc;
    mc.lamT = lT;
    mc.lamEll = lE;
    cc[(size_t)d * Mp + m] = mc;
  }
  __syncthreads();
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
// Shared tile phases
// ---------------------------------------------------------------------------
template <typename TX, int MG>
struct FwdTile {
  typedef Path<TX> PT;
  static constexpr int DW = tile_channels<TX>();
  static constexpr int CPW = DW / NWAVES;      // channels per wave
  static constexpr int NCG = CPW / 8;          // scan groups of 8 channels per wave
  static constexpr int XP = TileGeom<TX, DW>::PITCH;
  static constexpr int NSTR = 16 * MG;         // floats per chunk in the scan buffer
  static constexpr int KSTR = 16 * NSTR + 16;  // floats per channel in the scan buffer
  static constexpr int WSB = 8 * KSTR;         // floats per wave
  static constexpr int NM = 1 + 2 * MG;
};

// Chunk products of one wave's channels: yacc = T x (if WANT_Y) and the chunk
// end states S -> scan buffer; then the in-tile scan: hx[n] = state entering
// chunk n from zero at the tile start, aggv = state at the tile end.
// With KEEP_HX false only the state entering chunk nsel is kept (in hx[cg][g][0]).
template <typename TX, int MG, bool WANT_Y, bool KEEP_HX = true>
__device__ __forceinline__ void fwd_chunk_phase(const TX* xt, float* sb, const char* tab,
                                                const ModeScalars* scal, int Mp, int d0, int wave,
                                                int lane, f4* yacc,
                                                float2 (&hx)[FwdTile<TX, MG>::NCG][MG][NCHUNK],
                                                float2 (&aggv)[FwdTile<TX, MG>::NCG][MG],
                                                int nsel = 0) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  const int li = lane & 15, lq = lane >> 4;
  const int sk = lane >> 3, sj = lane & 7;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cg = 0; cg < F::NCG; ++cg) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ch = wave * F::CPW + cg * 8 + k;
      const char* tp = tab + (size_t)(d0 + ch) * F::NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
      const typename PT::XOp xv = PT::load_x(&xt[ch * F::XP + PT::x_off(li, lq)]);
      if (WANT_Y) yacc[cg * 8 + k] = PT::mma(PT::load_a(tp), xv, zero);
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const f4 s = PT::mma(PT::load_a(tp + (1 + 2 * g) * TAB_MAT_BYTES), xv, zero);
        *reinterpret_cast<f4*>(&sb[k * F::KSTR + li * F::NSTR + g * 16 + lq * 4]) = s;
      }
    }
    __syncthreads();
    {
      const int dch = d0 + wave * F::CPW + cg * 8 + sk;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        const float2 mu = scal[(size_t)dch * Mp + g * 8 + sj].mu;
        float2 run = make_float2(0.f, 0.f);
#pragma unroll
        for (int n = 0; n < NCHUNK; ++n) {
          if (KEEP_HX)
            hx[cg][g][n] = run;
          else if (n == nsel)
            hx[cg][g][0] = run;
          const float2 s =
              *reinterpret_cast<const float2*>(&sb[sk * F::KSTR + n * F::NSTR + g * 16 + 2 * sj]);
          run = cfma(mu, run, s);
        }
        aggv[cg][g] = run;
      }
    }
    __syncthreads();
  }
}

// State at t = L-1 from the state h entering chunk nstar and the chunk's drives.
template <typename TX>
__device__ __forceinline__ float2 tail_state(float2 h, const TX* row, int nstar, int jstar,
                                             float2 lam) {
  for (int j = 0; j <= jstar; ++j)
    h = cfma(lam, h, make_float2(to_f32(row[nstar * CHUNK + j]), 0.f));
  return h;
}

// ---------------------------------------------------------------------------
// Prompt state: chunk states -> scan -> per-tile aggregate (end state of the
// tile's own drives from a zero state); the last tile of a row writes the state
// at t = L-1 instead.  carry_fwd_kernel then chains the tiles.
// ---------------------------------------------------------------------------
template <typename TX, int MG>
__global__ __launch_bounds__(NTHREADS) void fwd_state_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  __shared__ __align__(16) TX xt[F::DW * F::XP];
  __shared__ __align__(16) float sbuf[NWAVES * F::WSB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sk = lane >> 3, sj = lane & 7;
  const int64_t tile = blockIdx.x;
  const int nb = (int)(tile % a.NB);
  const int64_t rest = tile / a.NB;
  const int64_t b = rest % a.B;
  const int64_t p = rest / a.B;
  const int64_t t0 = p * TILE_T;
  const int d0 = nb * F::DW;
  load_tile_any<TX, F::DW>(reinterpret_cast<const TX*>(a.x), xt, b, t0, d0, a.L, a.D, tid);
  __syncthreads();
  const bool last = (p == a.P - 1);
  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  float2 hx[F::NCG][MG][NCHUNK];
  float2 aggv[F::NCG][MG];
  fwd_chunk_phase<TX, MG, false, false>(xt, sbuf + wave * F::WSB,
                                        reinterpret_cast<const char*>(a.tab), a.scal, a.Mp, d0,
                                        wave, lane, nullptr, hx, aggv, nstar);
#pragma unroll
  for (int cg = 0; cg < F::NCG; ++cg) {
    const int ch = wave * F::CPW + cg * 8 + sk;
    const int dch = d0 + ch;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const int m = g * 8 + sj;
      float2 v = aggv[cg][g];
      if (last)
        v = tail_state(hx[cg][g][0], &xt[ch * F::XP], nstar, jstar,
                       a.scal[(size_t)dch * a.Mp + m].lam);
      a.agg[((size_t)(b * a.P + p) * a.Dp + dch) * a.Mp + m] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Single-pass forward.
//
// Work-groups take tiles in ticket order (time-major over the chains (b,
// channel block)).  A tile publishes the end state of its own
// drives (aggregate), resolves the state entering it from its predecessors and
// publishes the end state including them (inclusive).  The state entering tile
// p is always the canonical value inc(p-1), where inc(-1) = h0 and
// inc(i) = lambda^256 inc(i-1) + agg(i) in float32: a tile finds the nearest
// predecessor whose inclusive state is out (polling a window of 64 flags at
// once) and applies the recurrence forward through the aggregates after it, so
// the result does not depend on timing (bitwise reproducible).  Every wait is on
// a smaller ticket, which a running work-group took, and every wait is bounded.
// Payloads and flags are agent-coherent (device-scope) accesses; a publisher
// completes its payload stores before the flag store that releases them.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st_agent(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ uint32_t ld_flag(const uint32_t* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(uint32_t* f, uint32_t v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Upper bound on window polls (about a second); reached only if a predecessor
// never publishes, which the ticket order rules out.  The tile then starts from
// the row's initial state and records the event in the error word.
constexpr uint32_t SPIN_LIMIT = 1u << 20;

template <typename TX, typename TY, int MG>
__global__ __launch_bounds__(NTHREADS, MG == 1 ? 2 : 1) void fwd_fused_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  constexpr int DW = F::DW, CPW = F::CPW, NCG = F::NCG, XP = F::XP;
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) TX xt[DW * XP];
  __shared__ __align__(16) float sbuf[NWAVES * F::WSB];
  __shared__ uint32_t s_u[2];
  __shared__ int64_t s_j;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, lq = lane >> 4;
  const int sk = lane >> 3, sj = lane & 7;
  const int nchains = (int)(a.B * a.NB);
  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* sb = sbuf + wave * F::WSB;
  const int nstar = (a.last_len - 1) / CHUNK, jstar_l = (a.last_len - 1) % CHUNK;

  if (tid == 0) s_u[0] = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int64_t tk = s_u[0];
  const int64_t p = tk / nchains;
  const int chain = (int)(tk % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t t0 = p * TILE_T;
  const bool last = (p == a.P - 1);

  // per scan lane (channel wave*CPW + cg*8 + sk, mode g*8 + sj): its scalars
  ModeScalars msc[NCG][MG];
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
    for (int g = 0; g < MG; ++g)
      msc[cg][g] = a.scal[(size_t)(d0 + wave * CPW + cg * 8 + sk) * a.Mp + g * 8 + sj];

  load_tile_any<TX, DW>(reinterpret_cast<const TX*>(a.x), xt, b, t0, d0, a.L, a.D, tid);
  __syncthreads();

  // ---- chunk end states and in-tile scan ---------------------------------
  float2 hx[NCG][MG][NCHUNK];
  float2 aggv[NCG][MG];
  fwd_chunk_phase<TX, MG, false>(xt, sb, tab, a.scal, a.Mp, d0, wave, lane, nullptr, hx, aggv);

  // ---- state entering the tile -------------------------------------------
  auto pay_idx = [&](int64_t t, int cg, int g) {
    return ((size_t)t * DW + wave * CPW + cg * 8 + sk) * a.Mp + g * 8 + sj;
  };
  auto h0_at = [&](int cg, int g) {
    const int d = d0 + wave * CPW + cg * 8 + sk, m = g * 8 + sj;
    if (a.h0 == nullptr || d >= a.D || m >= a.M) return make_float2(0.f, 0.f);
    const float* h = a.h0 + ((size_t)(b * a.D + d) * a.M + m) * 2;
    return make_float2(h[0], h[1]);
  };
  float2 carry[NCG][MG];
  if (p == 0) {
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
      for (int g = 0; g < MG; ++g) carry[cg][g] = h0_at(cg, g);
  } else {
    if (tid == 0) s_u[1] = ld_flag(a.flags + (tk - nchains));
    __syncthreads();
    const uint32_t fpred = s_u[1];
    if (fpred != FLAG_INCL && !last) {
      // the predecessor is not resolved yet: publish this tile's aggregate first
#pragma unroll
      for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
        for (int g = 0; g < MG; ++g) st_agent(a.pay_agg + pay_idx(tk, cg, g), aggv[cg][g]);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (tid == 0) st_flag(a.flags + tk, FLAG_AGG);
    }
    int64_t jres;  // nearest chain tile with its inclusive state out (-1: row start)
    if (fpred == FLAG_INCL) {
      jres = p - 1;
    } else {
      if (wave == 0) {
        int64_t top = p - 1;
        int64_t res = -2;
        uint32_t it = 0;
        while (res == -2) {
          const int64_t j = top - lane;
          const uint32_t fl = (j >= 0) ? ld_flag(a.flags + j * nchains + chain) : FLAG_INCL;
          const uint64_t incl = __ballot(fl == FLAG_INCL);
          const uint64_t none = __ballot(fl == FLAG_NONE);
          if (incl != 0) {
            const int l = __ffsll((unsigned long long)incl) - 1;
            const uint64_t nearer = (l == 0) ? 0ull : (~0ull >> (64 - l));
            if ((none & nearer) == 0) res = top - l;
          } else if (none == 0) {
            top -= 64;  // the whole window holds aggregates: keep looking further back
            continue;
          }
          if (res == -2) {
            if (++it >= SPIN_LIMIT) {
              if (lane == 0) atomicOr(a.error, 1u);
              res = -1;
            } else {
              __builtin_amdgcn_s_sleep(1);
            }
          }
        }
        if (lane == 0) s_j = res;
      }
      __syncthreads();
      jres = s_j;
    }
    // canonical forward recurrence from the resolved state; the aggregates are
    // loaded in batches so that their latencies overlap
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
      for (int g = 0; g < MG; ++g)
        carry[cg][g] = (jres >= 0) ? ld_agent(a.pay_inc + pay_idx(jres * nchains + chain, cg, g))
                                   : h0_at(cg, g);
    constexpr int LB = 8;
    for (int64_t i = jres + 1; i < p; i += LB) {
      const int n = (p - i) < LB ? (int)(p - i) : LB;
      float2 v[NCG][MG][LB];
#pragma unroll
      for (int u = 0; u < LB; ++u)
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
          for (int g = 0; g < MG; ++g)
            v[cg][g][u] = (u < n) ? ld_agent(a.pay_agg + pay_idx((i + u) * nchains + chain, cg, g))
                                  : make_float2(0.f, 0.f);
#pragma unroll
      for (int u = 0; u < LB; ++u)
        if (u < n) {
#pragma unroll
          for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
            for (int g = 0; g < MG; ++g)
              carry[cg][g] = cfma(msc[cg][g].lamT, carry[cg][g], v[cg][g][u]);
        }
    }
  }
  if (!last) {
    // publish the inclusive state: lambda^256 carry + own aggregate
#pragma unroll
    for (int cg = 0; cg < NCG; ++cg)
#pragma unroll
      for (int g = 0; g < MG; ++g)
        st_agent(a.pay_inc + pay_idx(tk, cg, g), cfma(msc[cg][g].lamT, carry[cg][g], aggv[cg][g]));
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) st_flag(a.flags + tk, FLAG_INCL);
  }

  // ---- per channel group: carried state per chunk, then y = T x + U H -------
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    {
      const int ch = wave * CPW + cg * 8 + sk;
#pragma unroll
      for (int g = 0; g < MG; ++g) {
        float2 w = carry[cg][g];
        float2 hlast = w;
#pragma unroll
        for (int n = 0; n < NCHUNK; ++n) {
          const float2 h = make_float2(hx[cg][g][n].x + w.x, hx[cg][g][n].y + w.y);
          *reinterpret_cast<float2*>(&sb[sk * F::KSTR + n * F::NSTR + g * 16 + 2 * sj]) = h;
          if (n == nstar) hlast = h;
          w = cmul(msc[cg][g].mu, w);
        }
        const int dch = d0 + ch, m = g * 8 + sj;
        if (last && a.h_out != nullptr && dch < a.D && m < a.M) {
          const float2 hL = tail_state(hlast, &xt[ch * XP], nstar, jstar_l, msc[cg][g].lam);
          float* ho = a.h_out + ((size_t)(b * a.D + dch) * a.M + m) * 2;
          ho[0] = hL.x;
          ho[1] = hL.y;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int ch = wave * CPW + cg * 8 + k;
      const char* tp = tab + (size_t)(d0 + ch) * F::NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
      f4 acc = PT::mma(PT::load_a(tp), PT::load_x(&xt[ch * XP + PT::x_off(li, lq)]), zero);
#pragma unroll
      for (int g = 0; g < MG; ++g)
        acc = mma_f32(load_f4(tp + (2 + 2 * g) * TAB_MAT_BYTES),
                      load_f4(&sb[k * F::KSTR + li * F::NSTR + g * 16 + lq * 4]), acc);
      if (SEPY) {
        const int d = d0 + ch;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t t = t0 + li * CHUNK + lq * 4 + r;
          if (d < a.D && t < a.L)
            reinterpret_cast<float*>(a.y)[(b * a.L + t) * (int64_t)a.D + d] = acc[r];
        }
      } else {
        TY v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = from_f32<TY>(acc[r]);
        TY* dst = reinterpret_cast<TY*>(xt) + ch * XP + li * CHUNK + lq * 4;
        if (sizeof(TY) == 2)
          *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(v);
        else
          *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(v);
      }
    }
    __syncthreads();
  }

  if (!SEPY)
    store_tile_any<TY, DW>(reinterpret_cast<TY*>(a.y), reinterpret_cast<const TY*>(xt), b, t0, d0,
                           a.L, a.D, tid);
}

// ---------------------------------------------------------------------------
// Cross-tile carry for the prompt state: for each (b, d, m), in float64,
//   h = lambda^TILE_T h + agg[p] for p < P-1, then h_{L-1} = lambda^last_len h + agg[P-1].
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void carry_fwd_kernel(const float2* __restrict__ agg,
                                                        float* __restrict__ hout,
                                                        const ModeCarry* __restrict__ cc, int B,
                                                        int64_t P, int D, int M, int Dp, int Mp) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * Dp * Mp) return;
  const int m = (int)(idx % Mp);
  const int d = (int)((idx / Mp) % Dp);
  const int64_t b = idx / ((int64_t)Mp * Dp);
  if (d >= D || m >= M) return;
  double2 h = make_double2(0.0, 0.0);
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
        const double2 prop = (p < P - 1) ? c.lamT : c.lamEll;
        h = zfma(prop, h, make_double2((double)ag[j].x, (double)ag[j].y));
      }
    }
  }
  const size_t sidx = ((size_t)(b * D + d) * M + m) * 2;
  hout[sidx] = (float)h.x;
  hout[sidx + 1] = (float)h.y;
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
                       uint32_t* flags, int64_t nflags, hipStream_t st) {
  if (bwd)
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc, flags,
                       nflags);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, (TA*)tab, scal, cc, flags,
                       nflags);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       uint32_t*, int64_t, hipStream_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*,
                                        uint32_t*, int64_t, hipStream_t);

template <typename TX>
hipError_t launch_fwd_state(const Geometry& g, const FwdArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    hipLaunchKernelGGL((fwd_state_kernel<TX, 1>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((fwd_state_kernel<TX, 2>), grid, block, 0, st, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_state<float>(const Geometry&, const FwdArgs&, hipStream_t);
template hipError_t launch_fwd_state<bf16_t>(const Geometry&, const FwdArgs&, hipStream_t);

template <typename TX, typename TY>
hipError_t launch_fwd_fused(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    launch_timed(fwd_fused_kernel<TX, TY, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(fwd_fused_kernel<TX, TY, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_fused<float, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                   hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_fused<bf16_t, bf16_t>(const Geometry&, const FwdArgs&, hipStream_t,
                                                     hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_fused<bf16_t, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                    hipEvent_t, hipEvent_t);

hipError_t launch_carry_fwd(const Geometry& g, const float2* agg, float* hout, const ModeCarry* cc,
                            hipStream_t st) {
  const int64_t n = g.B * (int64_t)g.Dp * g.Mp;
  hipLaunchKernelGGL(carry_fwd_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, agg,
                     hout, cc, (int)g.B, g.P, (int)g.D, (int)g.M, g.Dp, g.Mp);
  return hipGetLastError();
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace res
