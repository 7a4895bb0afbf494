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
// Chunked form.  Chunk n of a 256-step tile is steps 16n .. 16n+15; (Q_n, R_n)
// is (q, rho) at step 16n from every drive at or after it, mu = lambda^16:
//   Q_n = Eq[n] + mu Q_{n+1},   R_n = Er[n] + mu (16 Q_{n+1} + R_{n+1})
//   Eq[n] = sum_i lambda^i dy[16n+i],   Er[n] = sum_i i lambda^i dy[16n+i]
//   dx[16n+j] = sum_{i>=j} K[i-j] dy[16n+i] + Re sum_m c lambda^(16-j) Q_{n+1}     (Tt, Ub)
//   W = lambda sum_n Xs[n] Q_{n+1} + sum_tau lambda^tau G[tau]
//   R = lambda sum_n ((Xs + Xw)[n] Q_{n+1} + Xs[n] R_{n+1}) + sum_tau tau lambda^tau G[tau]
//   Xs[n] = sum_k lambda^k x[16n+15-k],   Xw[n] = sum_k k lambda^k x[16n+15-k]
//   G[tau] = sum_n sum_j dy[16n+j+tau] x[16n+j]      (diagonal sums of P = DY X^T)
// The chunk sums of x weighted by lambda^(16-j) and (16-j) lambda^(16-j) that the
// carried states meet are lambda Xs and lambda (Xs + Xw): the tables of Eq and Er
// applied to x read backwards inside each chunk, with the factor lambda taken
// out of the sums.  Every product is a 16x16 MFMA per channel over the 16 chunks
// of a tile.
//
// Work decomposition.  A chain is one batch row and one block of 64-byte rows of
// channels (32 bf16 or 16 float channels); it is cut into segments of S tiles,
// one work-group each, four channels per wave.
//   bwd_state_kernel: the (Q, R) of each record segment's own drives at its
//     left edge (a segment, or half of one for float32 drives).
//   bwd_apply_kernel: the state entering the segment from the right (the later
//     segments' records folded in float64), then the tiles from right to left:
//     the products above, the chunk scan carried from tile to tile in
//     registers, dx, and the segment's partial sums of G, W and R.
//   bwd_reduce_kernel: fixed-order float64 sums of the partials, the gradients.
// The per-channel tables (Tt, Eq, Er, Ub) stay in registers for a whole segment.
#include "common.h"
#include "kernels.h"
#include "stream.h"

namespace res {

// Layout of the per-segment partial sums: [G(16) | per mode (W re, W im, R re, R im)]
// (W and R without the factor lambda of the carried part).
__host__ __device__ inline int part_stride(int Mp) { return 16 + 4 * Mp; }

// Chain block of the backward: 64-byte rows, four channels per wave.  The
// time-major LDS tile holds 16 groups of 16 rows (1 KB) filled by direct-to-LDS
// loads; each group is padded so that the 8-byte (bf16) or 16-byte (float)
// operand reads of 16 lanes from 16 groups fall on different banks.  Inside a
// row the four 16-byte pieces are swizzled: piece k of row t sits in slot
// k ^ ((t >> 2) & 3), so that 16 lanes reading one piece of the 16 rows of a
// group also meet 16 different slots.
template <typename TX>
struct BGeo {
  static constexpr int XE = (int)sizeof(TX);
  static constexpr int DW = 64 / XE;   // channels per block
  static constexpr int NW = DW / 4;    // waves
  static constexpr int NT = 64 * NW;
  static constexpr int ROWB = 64;
  static constexpr int GRP = 16 * ROWB + (XE == 2 ? 8 : 16);
  static constexpr int TB = 16 * GRP;  // bytes of a tile
  static constexpr int GPW = 16 / NW;  // row groups of a tile per wave
  // byte offset of channel byte cb (0..63) of step t
  __device__ static __forceinline__ int off(int t, int cb) {
    return (t >> 4) * GRP + (t & 15) * ROWB + ((((cb >> 4) ^ (t >> 2)) & 3) << 4) + (cb & 15);
  }
  // the piece slot of the 4 consecutive channels at ch0 in row group quarter s
  __device__ static __forceinline__ int slot(int ch0, int s) {
    return ((((ch0 * XE) >> 4) ^ s) & 3) * 16 + ((ch0 * XE) & 15);
  }
};

// Activation operands of channels ch0 .. ch0+3 in the MFMA B layout: lane (n, q)
// holds steps 16n + 4q + r, r = 0..3 (REV: steps 16n + 15 - 4q - r).
template <typename TX, bool REV>
__device__ __forceinline__ void bgather(const char* xt, int ch0, int n, int q, typename FPath<TX>::XOp (&v)[4]) {
  typedef BGeo<TX> G;
  const char* p = xt + n * G::GRP + G::slot(ch0, REV ? 3 - q : q);
  if constexpr (sizeof(TX) == 2) {
    typedef unsigned short us4 __attribute__((ext_vector_type(4)));
    us4 w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) w[r] = *reinterpret_cast<const us4*>(p + (REV ? 15 - 4 * q - r : 4 * q + r) * G::ROWB);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const us4 e = {w[0][c], w[1][c], w[2][c], w[3][c]};
      v[c] = __builtin_bit_cast(s4, e);
    }
  } else {
    f4 w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) w[r] = *reinterpret_cast<const f4*>(p + (REV ? 15 - 4 * q - r : 4 * q + r) * G::ROWB);
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = f4{w[0][c], w[1][c], w[2][c], w[3][c]};
  }
}

// Table products of the backward (the activation times a per-channel table).
//   bf16: split-bf16 on v_mfma_f32_16x16x32_bf16.  A table A (from float64) is
//     stored as Ah = bf16(A), Al = bf16(A - Ah), lane (i, q) holding
//     Ah[i][8q..8q+7] (q < 2) or Al[i][8(q-2)..8(q-2)+7] (q >= 2); lane (n, q) of
//     the activation operand holds steps 8 (q & 1) .. 8 (q & 1) + 7 of column n,
//     so that both halves of the 32-deep contraction meet the same steps and one
//     instruction gives (Ah + Al) x.
//   float: four v_mfma_f32_16x16x4_f32, 4 steps per lane (FPath<float>).
// The activation operand of channels ch0 .. ch0+3: lane (n, q) holds the steps of
// chunk n above (REV: step 16n + 15 - k in place of 16n + k).
template <typename TX> struct BPath;
template <> struct BPath<bf16_t> {
  typedef bf8 AOp;
  typedef bf8 XOp;
  __device__ static __forceinline__ AOp load_a_u4(uint4 u) { return __builtin_bit_cast(bf8, u); }
  __device__ static __forceinline__ f4 mma(const bf8& a, const bf8& b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  template <bool REV>
  __device__ static __forceinline__ void gather(const char* xt, int ch0, int n, int q, XOp (&v)[4]) {
    typedef BGeo<bf16_t> G;
    typedef unsigned short us4 __attribute__((ext_vector_type(4)));
    typedef unsigned short us8 __attribute__((ext_vector_type(8)));
    const char* p = xt + n * G::GRP;
    const int h = 8 * (q & 1);
    us4 w[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int row = REV ? 15 - h - r : h + r;
      w[r] = *reinterpret_cast<const us4*>(p + row * G::ROWB + G::slot(ch0, row >> 2));
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const us8 e = {w[0][c], w[1][c], w[2][c], w[3][c], w[4][c], w[5][c], w[6][c], w[7][c]};
      v[c] = __builtin_bit_cast(bf8, e);
    }
  }
};
template <> struct BPath<float> {
  typedef f4 AOp;
  typedef f4 XOp;
  __device__ static __forceinline__ AOp load_a_u4(uint4 u) { return __builtin_bit_cast(f4, u); }
  __device__ static __forceinline__ f4 mma(const f4& a, const f4& b, f4 c) { return mma_f32(a, b, c); }
  template <bool REV>
  __device__ static __forceinline__ void gather(const char* xt, int ch0, int n, int q, XOp (&v)[4]) {
    bgather<float, REV>(xt, ch0, n, q, v);
  }
};

// Operands contracting over the tile's chunks: lane (i, q) holds steps
// 16 (4q + r) + i, r = 0..3, of channels ch0 .. ch0+3.
template <typename TX>
__device__ __forceinline__ void cgather(const char* xt, int ch0, int i, int q, typename FPath<TX>::XOp (&v)[4]) {
  typedef BGeo<TX> G;
  const char* p = xt + i * G::ROWB + G::slot(ch0, i >> 2);
  if constexpr (sizeof(TX) == 2) {
    typedef unsigned short us4 __attribute__((ext_vector_type(4)));
    us4 w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) w[r] = *reinterpret_cast<const us4*>(p + (4 * q + r) * G::GRP);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const us4 e = {w[0][c], w[1][c], w[2][c], w[3][c]};
      v[c] = __builtin_bit_cast(s4, e);
    }
  } else {
    f4 w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) w[r] = *reinterpret_cast<const f4*>(p + (4 * q + r) * G::GRP);
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = f4{w[0][c], w[1][c], w[2][c], w[3][c]};
  }
}

// Outputs of channels ch0 .. ch0+3 in the MFMA D layout (lane (n, q) holds steps
// 16n + 4q + r) into the time-major tile.
template <typename TX>
__device__ __forceinline__ void bput4(char* xt, int ch0, int n, int q, const f4 (&acc)[4]) {
  typedef BGeo<TX> G;
  char* p = xt + n * G::GRP + 4 * q * G::ROWB + G::slot(ch0, q);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if constexpr (sizeof(TX) == 2) {
      typedef __bf16 bf4 __attribute__((ext_vector_type(4)));
      const bf4 v = {(__bf16)acc[0][r], (__bf16)acc[1][r], (__bf16)acc[2][r], (__bf16)acc[3][r]};
      *reinterpret_cast<bf4*>(p + r * G::ROWB) = v;
    } else {
      *reinterpret_cast<f4*>(p + r * G::ROWB) = f4{acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
    }
  }
}

// Direct-to-LDS load of the calling wave's row groups (g = wave + NW i) of a full
// tile: one 16-byte piece per lane, lane l taking row l / 4, piece l % 4.
template <typename TX>
__device__ __forceinline__ void bload(char* buf, const TX* src, int64_t b, int64_t t0, int d0, int64_t L, int D,
                                      int lane, int wave) {
  typedef BGeo<TX> G;
  const int64_t rowb = (int64_t)D * G::XE;
  const char* base = reinterpret_cast<const char*>(src) + ((b * L + t0) * D + d0) * G::XE;
  int ln = lane;
  asm volatile("" : "+v"(ln));
  // lane l fills slot l & 3 of row l >> 2: piece (l & 3) ^ quarter of the row
  const uint32_t loff = (uint32_t)((ln >> 2) * rowb) + (((ln & 3) ^ (ln >> 4)) & 3) * 16;
#pragma unroll
  for (int i = 0; i < G::GPW; ++i) {
    const int g = wave + G::NW * i;
    lds_dma16(base + (int64_t)(16 * g) * rowb, loff, buf + g * G::GRP);
  }
}

// Row stores of the calling wave's row groups of a full tile (the same groups
// as its loads), the LDS reads first, as two 8-byte halves.
template <typename TX>
__device__ __forceinline__ void bstore(TX* dst, const char* buf, int64_t b, int64_t t0, int d0, int64_t L, int D,
                                       int lane, int wave) {
  typedef BGeo<TX> G;
  const int64_t rowb = (int64_t)D * G::XE;
  char* base = reinterpret_cast<char*>(dst) + ((b * L + t0) * D + d0) * G::XE;
  int ln = lane;
  asm volatile("" : "+v"(ln));
  u32x4 v[G::GPW];
#pragma unroll
  for (int i = 0; i < G::GPW; ++i) {
    const uint2* s = reinterpret_cast<const uint2*>(buf + (wave + G::NW * i) * G::GRP + ln * 16);
    const uint2 u = s[0], w = s[1];
    v[i] = u32x4{u.x, u.y, w.x, w.y};
  }
  const uint32_t loff = (uint32_t)((ln >> 2) * rowb) + (((ln & 3) ^ (ln >> 4)) & 3) * 16;
#pragma unroll
  for (int i = 0; i < G::GPW; ++i) st_row16(base + (int64_t)(16 * (wave + G::NW * i)) * rowb, loff, v[i]);
}

// Element copy of a tile that is not full (every thread); zeros outside the tensor.
template <typename TX>
__device__ __forceinline__ void bcopy(char* buf, const TX* x, int64_t b, int64_t t0, int d0, int64_t L, int D,
                                      int tid) {
  typedef BGeo<TX> G;
  for (int idx = tid; idx < TILE_T * G::DW; idx += G::NT) {
    const int t = idx / G::DW, c = idx % G::DW;
    TX v = from_f32<TX>(0.f);
    if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
    *reinterpret_cast<TX*>(buf + G::off(t, c * G::XE)) = v;
  }
}

// Guarded element stores of a tile that is not full (every thread).
template <typename TX>
__device__ __forceinline__ void bstore_part(TX* y, const char* buf, int64_t b, int64_t t0, int d0, int64_t L,
                                            int D, int tid) {
  typedef BGeo<TX> G;
  for (int idx = tid; idx < TILE_T * G::DW; idx += G::NT) {
    const int t = idx / G::DW, c = idx % G::DW;
    if (t0 + t < L && d0 + c < D)
      y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TX*>(buf + G::off(t, c * G::XE));
  }
}

// The value of the other lane of a (re, im) lane pair (DPP quad_perm [1,0,3,2];
// every lane is written, so no old value is needed).
__device__ __forceinline__ float pair_val(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}
// A float moved across lanes by a DPP pattern.
template <int CTRL>
__device__ __forceinline__ float dppf(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// Sum over the 16 lanes of a row (every lane of the row gets it): quad pairs,
// quads, half-row mirror, row mirror.
__device__ __forceinline__ float row_sum16(float v) {
  v += dppf<0xB1>(v);
  v += dppf<0x4E>(v);
  v += dppf<0x141>(v);
  v += dppf<0x140>(v);
  return v;
}

// One chunk of the right-to-left scan on the lane's component (lane pair = re, im
// of one mode; the partner's values read by DPP quad_perm [1,0,3,2]):
//   products with the state (Q, R) = (Q_{n+1}, R_{n+1}):
//     b1o += xs Q, b1p += xs Q', b2o += xs R + xw Q, b2p += xs R' + xw Q'
//   then Q <- mur Q + mus Q' + eq, R <- mur t + mus t' + er, t = 16 Q + R
// (mus = -Im mu on the re lane, +Im mu on the im lane).  A DPP read needs two
// wait states after a vector write of its source: every DPP source here was
// written at least two instructions earlier inside this block or before it.
__device__ __forceinline__ void scan_step(float& Q, float& R, float xs, float xw, float eq, float er, float mur,
                                          float mus, float c16, float& b1o, float& b1p, float& b2o, float& b2p) {
  float t, qn, rn;
  asm volatile(
      "v_fmac_f32 %[b1o], %[Q], %[xs]\n\t"
      "v_fmac_f32 %[b2o], %[R], %[xs]\n\t"
      "v_fmac_f32 %[b2o], %[Q], %[xw]\n\t"
      "v_fmac_f32_dpp %[b1p], %[Q], %[xs] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %[b2p], %[Q], %[xw] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fmac_f32_dpp %[b2p], %[R], %[xs] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fma_f32 %[t], %[Q], %[c16], %[R]\n\t"
      "v_fma_f32 %[qn], %[mur], %[Q], %[eq]\n\t"
      "v_fmac_f32_dpp %[qn], %[Q], %[mus] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "v_fma_f32 %[rn], %[mur], %[t], %[er]\n\t"
      "v_fmac_f32_dpp %[rn], %[t], %[mus] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf"
      : [b1o] "+v"(b1o), [b1p] "+v"(b1p), [b2o] "+v"(b2o), [b2p] "+v"(b2p), [t] "=&v"(t), [qn] "=&v"(qn),
        [rn] "=&v"(rn)
      : [Q] "v"(Q), [R] "v"(R), [xs] "v"(xs), [xw] "v"(xw), [eq] "v"(eq), [er] "v"(er), [mur] "v"(mur),
        [mus] "v"(mus), [c16] "s"(c16));
  Q = qn;
  R = rn;
}

// z^e for e >= 0 by binary powering (float64).
__device__ __forceinline__ double2 zpow(double2 z, int64_t e) {
  double2 r = make_double2(1.0, 0.0);
  for (; e > 0; e >>= 1) {
    if (e & 1) r = zmul(r, z);
    z = zmul(z, z);
  }
  return r;
}
// z^e for 0 <= e < 16 by binary powering (float32).
__device__ __forceinline__ float2 cpow16(float2 z, int e) {
  float2 r = make_float2(1.f, 0.f);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if ((e >> i) & 1) r = cmul(r, z);
    z = cmul(z, z);
  }
  return r;
}

// Work-group -> (batch row, segment, channel block).  The two 64-byte halves of
// a 128-byte row (blocks 2k and 2k+1) go to work-groups 8 apart, which the
// dispatcher places on the same XCD (work-groups go round-robin over the 8
// XCDs), so that both halves of every line are served by one L2.  Work-groups
// past the last block or row have no task.
struct BwdTask {
  int64_t b;
  int seg, nb;
  bool valid;
};
__device__ __forceinline__ BwdTask bwd_task(const BwdArgs& a) {
  const unsigned x = blockIdx.x;
  const unsigned hf = (x >> 3) & 1u, v = (x >> 4) * 8u + (x & 7u);
  const unsigned npair = (unsigned)(a.NB + 1) / 2u;
  const unsigned rest = v / npair;
  BwdTask t;
  t.nb = (int)(2u * (v % npair) + hf);
  t.seg = (int)(rest % (unsigned)a.nseg);
  t.b = (int64_t)(rest / (unsigned)a.nseg);
  t.valid = t.nb < a.NB && t.b < a.B;
  return t;
}
inline unsigned bwd_grid(const BwdArgs& a) {
  const int64_t v = (int64_t)((a.NB + 1) / 2) * a.B * a.nseg;
  return (unsigned)(((v + 7) / 8) * 16);
}

// ---------------------------------------------------------------------------
// Segment records.  Work-group (chain, segment), tiles p0 .. p0 + nt - 1 from
// the last to the first, four channels per wave.  Lane (n, q) of a channel's
// products Eq, Er (MFMA D layout) holds modes 2q, 2q+1 of chunk n; it keeps the
// pair (Q_n, R_n) of chunk n summed over the tiles by Horner's rule,
//   R_n <- h (R_n + 256 Q_n) + Er_k[n],   Q_n <- h Q_n + Eq_k[n],   h = lambda^256,
// and the segment's (Q, rho) at its left edge is, at the end,
//   Q = sum_n mu^n Q_n,   rho = sum_n mu^n (R_n + 16 n Q_n),   mu = lambda^16
// (the 16 chunk lanes summed across the row).  NBUF tile buffers, the first
// NBUF tiles loaded at once and the tiles taken in pairs (one barrier per pair):
// eight for segments of up to eight tiles in flight at once, one
// work-group per compute unit; four for half-segments (float32 drives: the
// records are taken per half of a segment of the segment pass), two work-groups
// of four waves per compute unit, so that one's arithmetic overlaps the other's
// waits (bf16 work-groups have eight waves, and two of them per compute unit
// would leave 128 registers a lane: measured slower).
// ---------------------------------------------------------------------------
template <typename TX, int MG, int NBUF>
__global__ __launch_bounds__(BGeo<TX>::NT, NBUF == 8 ? 1 : BGeo<TX>::NW / 2) void bwd_state_kernel(BwdArgs a) {
  typedef BGeo<TX> G;
  typedef BPath<TX> PT;
  constexpr int NM = bwd_mats(MG);
  __shared__ __align__(16) char tb[NBUF][G::TB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 15, lq = lane >> 4;
  const BwdTask task = bwd_task(a);
  if (!task.valid) return;
  const int nb = task.nb, seg = task.seg;
  const int64_t b = task.b;
  const int d0 = nb * G::DW, ch0 = 4 * wave;
  const int64_t p0 = (int64_t)seg * a.S;
  const int nt = (int)(a.P - p0 < a.S ? a.P - p0 : a.S);
  const TX* dy = reinterpret_cast<const TX*>(a.dy);
  auto tile_full = [&](int64_t p) { return a.fast_io && (p + 1) * TILE_T <= a.L && d0 + G::DW <= a.D; };

  // the tables and mode constants first (ahead of the tile loads in the memory queues)
  const char* tab = reinterpret_cast<const char*>(a.tab);
  typename PT::AOp teq[MG][4], ter[MG][4];
  float2 hop[MG][4][2], mu[MG][4][2], aq[MG][4][2], ar[MG][4][2];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int d = d0 + ch0 + c;
    const char* tp = tab + (size_t)d * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      teq[g][c] = PT::load_a_u4(*reinterpret_cast<const uint4*>(tp + (1 + 3 * g) * TAB_MAT_BYTES));
      ter[g][c] = PT::load_a_u4(*reinterpret_cast<const uint4*>(tp + (2 + 3 * g) * TAB_MAT_BYTES));
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const ModeScalars& ms = a.scal[(size_t)d * a.Mp + 8 * g + 2 * lq + h];
        hop[g][c][h] = ms.lamT;
        mu[g][c][h] = ms.mu;
        aq[g][c][h] = make_float2(0.f, 0.f);
        ar[g][c][h] = aq[g][c][h];
      }
    }
  }

  uint32_t issued = 0, mark[NBUF];
  auto tile_of = [&](int k) { return p0 + nt - 1 - k; };
  // the first NBUF tiles at once (a whole segment of up to NBUF tiles)
#pragma unroll
  for (int k = 0; k < NBUF; ++k) {
    if (k < nt && tile_full(tile_of(k))) {
      bload<TX>(tb[k], dy, b, tile_of(k) * TILE_T, d0, a.L, a.D, lane, wave);
      issued += G::GPW;
    }
    mark[k] = issued;
  }
  // lambda^(16 n) of the lane's chunk, for the end
#pragma unroll
  for (int g = 0; g < MG; ++g)
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) mu[g][c][h] = cpow16(mu[g][c][h], ln);

  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  auto tile_records = [&](int u) {
    typename PT::XOp dyv[4];
    PT::template gather<false>(tb[u], ch0, ln, lq, dyv);
#pragma unroll
    for (int g = 0; g < MG; ++g) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const f4 eq = PT::mma(teq[g][c], dyv[c], zero);
        const f4 er = PT::mma(ter[g][c], dyv[c], zero);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float2 t = make_float2(fmaf(256.f, aq[g][c][h].x, ar[g][c][h].x),
                                       fmaf(256.f, aq[g][c][h].y, ar[g][c][h].y));
          ar[g][c][h] = cfma(hop[g][c][h], t, make_float2(er[2 * h], er[2 * h + 1]));
          aq[g][c][h] = cfma(hop[g][c][h], aq[g][c][h], make_float2(eq[2 * h], eq[2 * h + 1]));
        }
      }
    }
  };
  // tiles in pairs, one wait and one barrier per pair (the pair's two tiles in
  // order, so the sums are those of one tile at a time)
  for (int k = 0; k < nt; k += 2) {
    const bool two = k + 1 < nt;
    const int u0 = k & (NBUF - 1), u1 = (k + 1) & (NBUF - 1);
    if (!tile_full(tile_of(k))) bcopy<TX>(tb[u0], dy, b, tile_of(k) * TILE_T, d0, a.L, a.D, tid);
    if (two && !tile_full(tile_of(k + 1))) bcopy<TX>(tb[u1], dy, b, tile_of(k + 1) * TILE_T, d0, a.L, a.D, tid);
    // the pair's direct loads are in once the later tile's are (loads complete in order)
    wait_vmcnt((int)(issued - mark[two ? u1 : u0]));
    __syncthreads();
    // tiles k+NBUF-2 and k+NBUF-1 (those not loaded at the start) into the buffers
    // of tiles k-2 and k-1, which every wave has finished with
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kn = k + NBUF - 2 + i;
      if (kn >= NBUF && kn < nt) {
        const int un = kn & (NBUF - 1);
        if (tile_full(tile_of(kn))) {
          bload<TX>(tb[un], dy, b, tile_of(kn) * TILE_T, d0, a.L, a.D, lane, wave);
          issued += G::GPW;
        }
        mark[un] = issued;
      }
    }
    tile_records(u0);
    if (two) tile_records(u1);
  }

  const size_t rec = (size_t)(b * a.nseg + seg) * a.Dp;
  const float s16 = 16.f * (float)ln;
#pragma unroll
  for (int g = 0; g < MG; ++g) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = d0 + ch0 + c;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float2 w = mu[g][c][h];
        const float2 q = cmul(w, aq[g][c][h]);
        const float2 r = cmul(w, make_float2(fmaf(s16, aq[g][c][h].x, ar[g][c][h].x),
                                             fmaf(s16, aq[g][c][h].y, ar[g][c][h].y)));
        const float4 v = make_float4(row_sum16(q.x), row_sum16(q.y), row_sum16(r.x), row_sum16(r.y));
        if (ln == 0) a.agg[(rec + d) * a.Mp + 8 * g + 2 * lq + h] = v;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Segment pass.  Work-group (chain, segment), tiles from the segment's last to
// its first; three buffer pairs (x, dy), two tiles ahead.  Per tile and wave
// (channels ch0 .. ch0+3):
//   products: P += DY X^T, dx = Tt dy, and per mode group Eq, Er (of dy), Xs, Xw
//     (of x read backwards) in the transposed layout, moved by lane swaps so
//     that lane (component i, channel c) holds chunks 0..15 of component i;
//   scan: from the state entering the tile on the right, chunk 15 down to 0, with
//     the partner component of each complex product read across the lane pair;
//     the states Q_{n+1} go through a per-wave LDS block to the MFMA layout for
//     dx += Ub Q, and the sums for W and R accumulate per lane;
//   dx replaces the wave's own dy columns of the tile; the rows leave after the
//   next tile's barrier (one barrier per tile), and each wave then loads tile
//   j+2 into the row groups it has just read out.
// The state at the tile's left edge carries to the next tile in registers.
// ---------------------------------------------------------------------------
constexpr int BH_P = 20;               // floats per chunk row of the state block (16 + 4 of bank offset)
constexpr int BH_K = 16 * BH_P + 4;    // floats per channel of the state block
static_assert(4 * BH_K >= 4 * 16 * 17, "the state block also holds the P dump");

template <typename TX, int MG>
__global__ __launch_bounds__(BGeo<TX>::NT, 1) void bwd_apply_kernel(BwdArgs a) {
  typedef BGeo<TX> G;
  typedef BPath<TX> PT;
  typedef FPath<TX> UT;
  typedef typename PT::XOp XOp;
  constexpr int NBUF = 3;
  constexpr int NM = bwd_mats(MG);
  __shared__ __align__(16) char xb[NBUF][G::TB];
  __shared__ __align__(16) char yb[NBUF][G::TB];
  __shared__ __align__(16) float hb[G::NW * 4 * BH_K];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ln = lane & 15, lq = lane >> 4;
  const BwdTask task = bwd_task(a);
  if (!task.valid) return;
  const int nb = task.nb, seg = task.seg;
  const int64_t b = task.b;
  const int d0 = nb * G::DW, ch0 = 4 * wave;
  const int64_t p0 = (int64_t)seg * a.S;
  const int nt = (int)(a.P - p0 < a.S ? a.P - p0 : a.S);
  const int64_t plast = p0 + nt - 1;
  const TX* x = reinterpret_cast<const TX*>(a.x);
  const TX* dy = reinterpret_cast<const TX*>(a.dy);
  TX* dx = reinterpret_cast<TX*>(a.dx);
  auto tile_full = [&](int64_t p) { return a.fast_io && (p + 1) * TILE_T <= a.L && d0 + G::DW <= a.D; };
  auto load = [&](int u, int64_t p) {
    bload<TX>(xb[u], x, b, p * TILE_T, d0, a.L, a.D, lane, wave);
    bload<TX>(yb[u], dy, b, p * TILE_T, d0, a.L, a.D, lane, wave);
  };

  // Loads of the tables, the mode constants and the first records of the later
  // segments go out first, then the first two tiles; the values are taken up
  // after the tile loads are issued.
  const char* tab = reinterpret_cast<const char*>(a.tab);
  uint4 rtt[4], rteq[MG][4], rter[MG][4];
  f4 rub[MG][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const char* tp = tab + (size_t)(d0 + ch0 + c) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
    rtt[c] = *reinterpret_cast<const uint4*>(tp);
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      rteq[g][c] = *reinterpret_cast<const uint4*>(tp + (1 + 3 * g) * TAB_MAT_BYTES);
      rter[g][c] = *reinterpret_cast<const uint4*>(tp + (2 + 3 * g) * TAB_MAT_BYTES);
      rub[g][c] = load_f4(tp + (3 + 3 * g) * TAB_MAT_BYTES);
    }
  }
  // scan lane (component ln, channel lq): channel sd, mode 8 g + ln / 2
  const int sd = d0 + ch0 + lq;
  const int hc = ln & 1;
  constexpr int FB = 8;
  float2 rmu[MG];
  double2 rlt[MG];
  float4 A[MG][FB];
  // the records are per record segment (a.sf of them per segment of this pass,
  // a.Ss tiles each); the later ones start at record segment jlo
  const int jlo = (seg + 1) * a.sf;
  auto records = [&](int g, int j1) {
#pragma unroll
    for (int i = 0; i < FB; ++i) {
      const int j = j1 - i >= jlo ? j1 - i : j1;  // past the first later record: any valid record, unused
      A[g][i] = a.agg[((size_t)(b * a.nss + j) * a.Dp + sd) * a.Mp + 8 * g + (ln >> 1)];
    }
  };
#pragma unroll
  for (int g = 0; g < MG; ++g) {
    const size_t im = (size_t)sd * a.Mp + 8 * g + (ln >> 1);
    rmu[g] = a.scal[im].mu;
    rlt[g] = a.cc[im].lamT;
    if (a.nss - 1 >= jlo) records(g, a.nss - 1);
  }

  uint32_t issued = 0, mark[NBUF] = {0u, 0u, 0u};
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (j < nt && tile_full(plast - j)) {
      load(j, plast - j);
      issued += 2 * G::GPW;
    }
    mark[j] = issued;
  }

  typename PT::AOp tt[4], teq[MG][4], ter[MG][4];
  typename UT::UOp ub[MG][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    tt[c] = PT::load_a_u4(rtt[c]);
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      teq[g][c] = PT::load_a_u4(rteq[g][c]);
      ter[g][c] = PT::load_a_u4(rter[g][c]);
      ub[g][c] = UT::u_op(rub[g][c]);
    }
  }
  float mur[MG], mus[MG], Qc[MG], Rc[MG];
#pragma unroll
  for (int g = 0; g < MG; ++g) {
    mur[g] = rmu[g].x;
    mus[g] = hc ? rmu[g].y : -rmu[g].y;
    // the state entering the segment from the right: the later records j, right
    // to left, C <- (lambda^(256 Ss) C_Q, lambda^(256 Ss) (C_R + 256 Ss C_Q)) + A_j
    const double2 hop = zpow(rlt[g], a.Ss);
    const double span = (double)TILE_T * (double)a.Ss;
    double2 CQ = make_double2(0.0, 0.0), CR = CQ;
    for (int j1 = a.nss - 1; j1 >= jlo; j1 -= FB) {
      if (j1 != a.nss - 1) records(g, j1);
#pragma unroll
      for (int i = 0; i < FB; ++i) {
        if (j1 - i >= jlo) {
          const double2 t = make_double2(fma(span, CQ.x, CR.x), fma(span, CQ.y, CR.y));
          CR = zfma(hop, t, make_double2(A[g][i].z, A[g][i].w));
          CQ = zfma(hop, CQ, make_double2(A[g][i].x, A[g][i].y));
        }
      }
    }
    Qc[g] = (float)(hc ? CQ.y : CQ.x);
    Rc[g] = (float)(hc ? CR.y : CR.x);
  }

  float b1o[MG], b1p[MG], b2o[MG], b2p[MG];
#pragma unroll
  for (int g = 0; g < MG; ++g) b1o[g] = b1p[g] = b2o[g] = b2p[g] = 0.f;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  f4 pacc[4] = {zero, zero, zero, zero};
  float* hw = hb + wave * 4 * BH_K;
  const float c16 = __builtin_amdgcn_readfirstlane(16.f);

  for (int j = 0; j < nt; ++j) {
    const int u = j % NBUF;
    const int64_t p = plast - j;
    if (tile_full(p)) {
      wait_vmcnt((int)(issued - mark[u]));
    } else {
      bcopy<TX>(xb[u], x, b, p * TILE_T, d0, a.L, a.D, tid);
      bcopy<TX>(yb[u], dy, b, p * TILE_T, d0, a.L, a.D, tid);
    }
    // tile j is in; every wave is done with tile j-1 (its x read, its dx written)
    __syncthreads();
    // the rows of tile j-1 and the load of tile j+2: the upper half of the waves
    // issues them before the products, the lower half after, so that the two
    // waves of a SIMD run their matrix and vector phases out of step
    auto memory = [&]() {
    if (j >= 1) {
      // the rows of dx of tile j-1, then tile j+2 into the same buffers (each
      // wave loads the row groups it has just read out)
      const int up = (j - 1) % NBUF;
      if (tile_full(p + 1)) {
        bstore<TX>(dx, yb[up], b, (p + 1) * TILE_T, d0, a.L, a.D, lane, wave);
        issued += G::GPW;
      } else {
        bstore_part<TX>(dx, yb[up], b, (p + 1) * TILE_T, d0, a.L, a.D, tid);
        __syncthreads();  // every thread read the whole tile
      }
    }
    if (j + 2 < nt) {
      const int u2 = (j + 2) % NBUF;
      if (tile_full(p - 2)) {
        load(u2, p - 2);
        issued += 2 * G::GPW;
      }
      mark[u2] = issued;
    }
    };
    const bool mem_first = wave >= G::NW / 2 || !tile_full(p + 1) || j == 0;
    if (mem_first) memory();

    const char* xt = xb[u];
    char* yt = yb[u];
    f4 dxa[4];
    XOp dyv[4], xrv[4];
    {
      typename FPath<TX>::XOp dyc[4], xc[4];
      cgather<TX>(yt, ch0, ln, lq, dyc);
      cgather<TX>(xt, ch0, ln, lq, xc);
      PT::template gather<false>(yt, ch0, ln, lq, dyv);
      PT::template gather<true>(xt, ch0, ln, lq, xrv);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        pacc[c] = mma_k16_act(dyc[c], xc[c], pacc[c]);
        dxa[c] = PT::mma(tt[c], dyv[c], zero);
      }
    }
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      float Eq[16], Er[16], Xs[16], Xw[16];
      {
        f4 R[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) R[c] = PT::mma(dyv[c], teq[g][c], zero);
        lanes_to_chunks(R, Eq);
#pragma unroll
        for (int c = 0; c < 4; ++c) R[c] = PT::mma(dyv[c], ter[g][c], zero);
        lanes_to_chunks(R, Er);
#pragma unroll
        for (int c = 0; c < 4; ++c) R[c] = PT::mma(xrv[c], teq[g][c], zero);
        lanes_to_chunks(R, Xs);
#pragma unroll
        for (int c = 0; c < 4; ++c) R[c] = PT::mma(xrv[c], ter[g][c], zero);
        lanes_to_chunks(R, Xw);
      }
      float Q = Qc[g], Rr = Rc[g];
#pragma unroll
      for (int n = 15; n >= 0; --n) {
        // (Q, Rr) = (Q_{n+1}, R_{n+1}): to the state block, then the chunk
        hw[lq * BH_K + n * BH_P + ln] = Q;
        scan_step(Q, Rr, Xs[n], Xw[n], Eq[n], Er[n], mur[g], mus[g], c16, b1o[g], b1p[g], b2o[g], b2p[g]);
      }
      Qc[g] = Q;
      Rc[g] = Rr;
      wave_lds_order();
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const f4 h = *reinterpret_cast<const f4*>(&hw[c * BH_K + ln * BH_P + 4 * lq]);
        dxa[c] = UT::mma_u(ub[g][c], h, dxa[c]);
      }
      wave_lds_order();
    }
    // dx in place of the wave's own dy columns (read above by this wave only)
    bput4<TX>(yt, ch0, ln, lq, dxa);
    if (!mem_first) memory();
  }
  __syncthreads();
  {
    const int up = (nt - 1) % NBUF;
    if (tile_full(p0))
      bstore<TX>(dx, yb[up], b, p0 * TILE_T, d0, a.L, a.D, lane, wave);
    else
      bstore_part<TX>(dx, yb[up], b, p0 * TILE_T, d0, a.L, a.D, tid);
  }

  // (Q, rho) at t = 0
  if (seg == 0) {
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      float* q = reinterpret_cast<float*>(a.q0 + ((size_t)b * a.Dp + sd) * a.Mp + 8 * g + (ln >> 1));
      q[hc] = Qc[g];
      q[2 + hc] = Rc[g];
    }
  }
  // partial sums of the segment: W = B1, R = B1 + B2 per mode from the lane pair
  // (re lane: own products minus the partner's, im lane: cross products added)
  const size_t rec = (size_t)(b * a.nseg + seg) * a.Dp;
  const int ps = part_stride(a.Mp);
#pragma unroll
  for (int g = 0; g < MG; ++g) {
    const float o1 = swap_pair(b1o[g]), p1 = swap_pair(b1p[g]);
    const float o2 = swap_pair(b2o[g]), p2 = swap_pair(b2p[g]);
    if (hc == 0) {
      const float wr = b1o[g] - o1, wi = b1p[g] + p1;
      const float4 v = make_float4(wr, wi, wr + (b2o[g] - o2), wi + (b2p[g] + p2));
      *reinterpret_cast<float4*>(a.part + (rec + sd) * ps + 16 + 4 * (8 * g + (ln >> 1))) = v;
    }
  }
  // G[tau]: P (lane (j, q) holds P[4q + r][j]) through the state block, then the
  // diagonal sums by lane (tau, channel)
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int r = 0; r < 4; ++r) hw[c * 272 + (4 * lq + r) * 17 + ln] = pacc[c][r];
  }
  wave_lds_order();
  float sg = 0.f;
  for (int jj = 0; jj + ln < 16; ++jj) sg += hw[lq * 272 + (jj + ln) * 17 + jj];
  a.part[(rec + sd) * ps + ln] = sg;
}

// ---------------------------------------------------------------------------
// Fixed-order reduction of the per-segment partials (float64), one block per channel d:
//   W = lambda sum_segments W' + sum_tau lambda^tau G[tau] + sum_b lambda q0 h0
//   R = lambda sum_segments R' + sum_tau tau lambda^tau G[tau] + sum_b lambda (q0 + rho0) h0
//   damp = Re(e^{i phi} W), dphase = -Im(c W), dgamma = -Re(c R), domega = -Im(c R)
//   dh0[b,d,m] = (Re(c lambda q0), -Im(c lambda q0))
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bwd_reduce_kernel(
    const float* __restrict__ part, const float4* __restrict__ q0, const ModeCarry* __restrict__ cc,
    const float* __restrict__ h0, float* __restrict__ dgamma, float* __restrict__ domega,
    float* __restrict__ damp, float* __restrict__ dphase, float* __restrict__ dh0, int B,
    int64_t nrows, int D, int M, int Dp, int Mp) {
  // One block per channel d.  The ps columns of the partial rows of d are summed
  // over the nrows (batch row, segment) records in float64: thread (row group rg,
  // column col) takes records rg, rg + NRG, ... in batches of eight loads issued
  // together (predicated past the last record), then the row groups are added
  // in order.  The order is fixed, so the result is bitwise reproducible.
  const int d = blockIdx.x;
  const int ps = part_stride(Mp);
  const int nrg = blockDim.x / ps;
  __shared__ double s_acc[256];
  __shared__ double s_col[16 + 4 * MODES_PER_GROUP * MG_MAX];
  {
    const int col = threadIdx.x % ps, rg = threadIdx.x / ps;
    double acc = 0.0;
    if (rg < nrg) {
      for (int64_t bp = rg; bp < nrows; bp += 8 * (int64_t)nrg) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int64_t r = bp + u * (int64_t)nrg;
          v[u] = r < nrows ? part[((size_t)r * Dp + d) * ps + col] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc += v[u];
      }
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
  // lambda, c and e^{i phase} of the mode, from the parameter tables (float64)
  const ModeCarry& mc = cc[(size_t)d * Mp + m];
  const double2 lam = mc.lam1, ph = mc.ephi;
  const double cp = ph.x, sp = ph.y;
  // the carried parts, times lambda
  const double2 W0 = zmul(lam, make_double2(s_col[16 + 4 * m], s_col[16 + 4 * m + 1]));
  const double2 R0 = zmul(lam, make_double2(s_col[16 + 4 * m + 2], s_col[16 + 4 * m + 3]));
  double Wr = W0.x, Wi = W0.y, Rr = R0.x, Ri = R0.y;
  // the taps: lambda^tau by successive products (float64)
  double2 pt = make_double2(1.0, 0.0);
#pragma unroll
  for (int t = 0; t < 16; ++t) {
    const double Gt = s_col[t];
    Wr = fma(pt.x, Gt, Wr);
    Wi = fma(pt.y, Gt, Wi);
    Rr = fma(t * pt.x, Gt, Rr);
    Ri = fma(t * pt.y, Gt, Ri);
    pt = zmul(pt, lam);
  }
  const double2 c = mc.c;
  const double2 cl = zmul(c, lam);
  for (int b = 0; (h0 != nullptr || dh0 != nullptr) && b < B; ++b) {
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
  const double2 cW = zmul(c, make_double2(Wr, Wi));
  const double2 cR = zmul(c, make_double2(Rr, Ri));
  damp[idx] = (float)(cp * Wr - sp * Wi);  // Re(e^{i phi} W)
  dphase[idx] = (float)(-cW.y);
  dgamma[idx] = (float)(-cR.x);
  domega[idx] = (float)(-cR.y);
}

// ---------------------------------------------------------------------------
int bwd_segments(int64_t nchains, int64_t P, int num_cus) {
  // about one work-group per compute unit, at least one tile per segment
  int64_t n = num_cus > nchains ? num_cus / nchains : 1;
  if (n > P) n = P;
  if (n < 1) n = 1;
  return (int)n;
}

template <typename TX>
hipError_t launch_bwd(const BwdArgs& a, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  typedef BGeo<TX> G;
  const dim3 grid(bwd_grid(a)), block(G::NT);
  const bool mg1 = a.Mp == MODES_PER_GROUP;
  if (a.nseg > 1) {
    // the record pass over its own segmentation (a.nss segments of a.Ss tiles)
    BwdArgs sa = a;
    sa.nseg = a.nss;
    sa.S = a.Ss;
    const dim3 sgrid(bwd_grid(sa));
    if (sizeof(TX) == 4 && a.sf == 2 && mg1) {
      hipLaunchKernelGGL((bwd_state_kernel<float, 1, 4>), sgrid, block, 0, st, sa);
    } else {
      if (mg1)
        hipLaunchKernelGGL((bwd_state_kernel<TX, 1, 8>), sgrid, block, 0, st, sa);
      else
        hipLaunchKernelGGL((bwd_state_kernel<TX, 2, 8>), sgrid, block, 0, st, sa);
    }
  }
  if (mg1)
    launch_timed(bwd_apply_kernel<TX, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(bwd_apply_kernel<TX, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_bwd<float>(const BwdArgs&, hipStream_t, hipEvent_t, hipEvent_t);
template hipError_t launch_bwd<bf16_t>(const BwdArgs&, hipStream_t, hipEvent_t, hipEvent_t);

hipError_t launch_bwd_reduce(const Geometry& g, int nseg, const float* part, const float4* q0,
                             const ModeCarry* cc, const float* h0, float* dgamma, float* domega,
                             float* damp, float* dphase, float* dh0, hipStream_t st) {
  hipLaunchKernelGGL(bwd_reduce_kernel, dim3((unsigned)g.D), dim3(256), 0, st, part, q0, cc, h0, dgamma,
                     domega, damp, dphase, dh0, (int)g.B, g.B * (int64_t)nseg, (int)g.D, (int)g.M, g.Dp, g.Mp);
  return hipGetLastError();
}

}  // namespace res
