// Internal launch interface between the C ABI (api.hip) and the kernel files.
#pragma once

#include <hip/hip_ext.h>

#include "common.h"

namespace res {

enum { MODE_STATE = 0, MODE_APPLY = 1 };

// Mixer epilogue: limits and the block of rows of the parameter sums
constexpr int EPI_H_MAX = 32;   // heads
constexpr int EPI_K_MAX = 16;   // local-path taps
constexpr int EPI_ROWS = 64;    // rows per block partial
// floats of block partials (then H*H float64 terms) in the epilogue backward workspace
inline int64_t epi_part_floats(int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K) {
  const int64_t nblk = B * ((L + EPI_ROWS - 1) / EPI_ROWS);
  const int64_t P = H * H + H * dh + H * dh * K;
  return (nblk * P + 1) & ~(int64_t)1;  // even, so the float64 terms that follow are 8-byte aligned
}
inline size_t epi_workspace_bytes(int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K) {
  return (size_t)epi_part_floats(B, L, H, dh, K) * sizeof(float) + (size_t)(H * H) * sizeof(double);
}

// LDS tile buffers of the single-kernel forward work-group, by activation size
// (bf16: 16 waves, 4 buffers; float32: 8 waves, 3 buffers)
constexpr int seg_bufs(int elem_bytes) { return elem_bytes == 2 ? 4 : 3; }


struct FwdArgs {
  const void* x;
  void* y;           // null for the prompt state
  int64_t B, L;
  int D, M;
  int NB, Dp, Mp;
  int64_t P;
  int last_len;
  int fast_io;       // x and y 16-byte aligned and D * element size a multiple of 16
  const void* tab;
  const ModeScalars* scal;
  const ModeCarry* cc;
  const float* h0;   // [B][D][M][2] or null
  float* h_out;      // [B][D][M][2] or null: state at t = L-1
  void* agg;         // per tile [DW * Mp] float4: half-tile end states (A_0, A_1)
  void* car;         // per tile [DW * Mp] float4: entry states of both halves (null: none)
  float2* alast;     // [B][Dp][Mp]: state at t = L-1 from a zero start at the last tile
};

// Single-pass forward (M <= 8): problem, parameters and the workspace regions.
// A published segment state is a set of 64-bit words, each a float (low half)
// and the call's tag, epoch + 1 (high half); hdr[1] holds the epoch.
// Tile-to-tile chains (2 to 4 work-groups per chain) pass each tile's inclusive
// end state to the next tile through a ring of STREAM_RING slots per chain; a
// slot is written again only after the tile that read it has published its own
// state, so any ring length is safe.  The ring is laid out for at most
// STREAM_RING_CHAINS chains (more chains leave at most one work-group each on a
// 256-CU device).
constexpr int STREAM_RING = 4;
constexpr int64_t STREAM_RING_CHAINS = 128;

struct StreamArgs {
  const void* x;
  void* y;
  int64_t B, L;
  int D, M;
  int NB;              // channel blocks of DW channels
  int nchains;         // B * NB
  int64_t P;           // tiles per chain
  int last_len;        // valid steps of a chain's last tile
  int fast_io;         // x and y 16-byte aligned and rows a multiple of 16 bytes
  const float* gamma;
  const float* omega;
  const float* amp;
  const float* phase;
  const float* h0;     // [B][D][M][2] or null
  float* h_out;        // [B][D][M][2] or null
  uint32_t* hdr;       // [0] status (bit 0: a wait gave up, bit 1: stale counters), [1] epoch,
                       // [2] finished chains, [4] a wait of this call gave up
  uint32_t* chainw;    // [nchains][4]: next ticket, arrived work-groups, segment order (0 open,
                       // 1 static, 2 tickets), finished work-groups
  uint64_t* agg;       // [nchains][G][8 waves][64][DW / 32] published state of each segment
                       // (float | tag << 32 per word); laid out for up to P segments
  uint64_t* ring;       // [nchains][STREAM_RING][8 waves][64][DW / 32] I of recent tiles, or null:
                        // no tile-to-tile chains
};

// Backward (M <= 16).  A chain is one batch row and one block of DW channels
// (64-byte rows: 32 bf16 or 16 float channels), cut into nseg segments of S
// tiles (the last may be shorter), one work-group per segment.
struct BwdArgs {
  const void* x;
  const void* dy;
  void* dx;
  int64_t B, L;
  int D, M;
  int NB;               // channel blocks of the backward
  int Dp, Mp;           // padded channels and modes (record strides)
  int64_t P;            // tiles per row
  int64_t S;            // tiles per segment
  int nseg;             // segments per row
  int64_t Ss;           // tiles per record segment (the record pass's own segmentation)
  int nss;              // record segments per row
  int sf;               // record segments per segment (S = sf Ss; 1 or 2)
  int fast_io;          // x, dy and dx 16-byte aligned and rows a multiple of 16 bytes
  const void* tab;
  const ModeScalars* scal;
  const ModeCarry* cc;
  float4* agg;          // [B][nss][Dp][Mp]: (Q, rho) of a record segment's own drives at its left edge
  float* part;          // [B][nseg][Dp][16 + 4 Mp]: partial sums of G, W and R per segment
  float4* q0;           // [B][Dp][Mp]: (Q, rho) at t = 0
};

template <typename TA>
hipError_t launch_prep(const Geometry& g, const float* gamma, const float* omega, const float* amp,
                       const float* phase, bool bwd, void* tab, ModeScalars* scal, ModeCarry* cc,
                       hipStream_t st);

template <typename TX>
hipError_t launch_fwd_agg(const Geometry& g, const FwdArgs& a, hipStream_t st,
                          hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

hipError_t launch_fwd_carry(const Geometry& g, const FwdArgs& a, hipStream_t st);

// Work-groups per call of the single-pass forward, and its launch.
int fwd_stream_grid(int64_t nchains, int64_t P, int num_cus);
template <typename TX, typename TY>
hipError_t launch_fwd_stream(const StreamArgs& a, int grid, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1);

template <typename TX, typename TY>
hipError_t launch_fwd_apply(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1);

// Launch with optional start/stop events recorded around this one kernel.
template <typename K, typename... Args>
inline void launch_timed(K kernel, dim3 grid, dim3 block, hipStream_t st, hipEvent_t ev0,
                         hipEvent_t ev1, Args... args) {
  if (ev0 != nullptr)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, ev0, ev1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st);

template <typename TX, typename TY>
hipError_t launch_decode(int64_t B, int64_t D, int64_t M, const void* x, void* y,
                         const float* gamma, const float* omega, const float* amp,
                         const float* phase, float* state, hipStream_t st);
const char* launch_grouped_linear(const void* x, const void* W, void* y, int64_t N, int64_t d_in, int64_t d_out,
                                  int64_t G, bool bf16, hipStream_t st);
// MFMA grouped projection (proj.hip): one or two weights (W1 null for one) over
// the same x; shapes and alignments the kernel takes, else the library GEMM
bool grouped_proj_supported(const void* x, const void* W0, const void* W1, const void* y0, const void* y1,
                            int64_t d_in, int64_t d_out, int64_t G, bool bf16);
hipError_t launch_grouped_proj(const void* x, const void* W0, const void* W1, void* y0, void* y1, int64_t N,
                               int64_t d_in, int64_t d_out, int64_t G, bool bf16, int num_cus, hipStream_t st);
bool grouped_dgrad_supported(int n, const void* const* dy, const void* const* W, const void* dx, int64_t d_in,
                             int64_t d_out, int64_t G, bool bf16);
hipError_t launch_grouped_dgrad(int n, const void* const* dy, const void* const* W, void* dx, int64_t N, int64_t d_in,
                                int64_t d_out, int64_t G, bool bf16, bool accumulate, int num_cus, hipStream_t st);
int grouped_wgrad_blocks(int n, int nout, int64_t d_in, int64_t d_out, int64_t G, bool bf16);
int64_t grouped_wgrad_grid(int64_t N, int n);
hipError_t launch_grouped_wgrad(int n, const void* x, const void* const* dy, const int* out, float* dW0, float* dW1,
                                int64_t N, int64_t d_in, int64_t d_out, int64_t G, bool accumulate, float* part,
                                hipStream_t st);
const char* launch_grouped_linear_bwd_data(const void* dy, const void* W, void* dx, int64_t N, int64_t d_in,
                                           int64_t d_out, int64_t G, bool bf16, bool accumulate, hipStream_t st);
const char* launch_grouped_linear_bwd_weight(const void* x, const void* dy, float* dW, int64_t N, int64_t d_in,
                                             int64_t d_out, int64_t G, bool bf16, bool accumulate, hipStream_t st);
hipError_t launch_block_diag(const void* W, void* Wd, int64_t d_in, int64_t d_out, int64_t G, bool bf16,
                             hipStream_t st);
constexpr int64_t SPLITK_TARGET = 64;     // partial products of the split-K weight gradient
constexpr int64_t SPLITK_MIN_ROWS = 256;  // rows per partial at least
int64_t splitk_rows(int64_t N);
int64_t splitk_parts(int64_t N);
const char* launch_grouped_linear_bwd_weight_splitk(const void* x, const void* dy, float* dW, int64_t N,
                                                    int64_t d_in, int64_t d_out, int64_t G, bool bf16,
                                                    bool accumulate, float* P, hipStream_t st);
hipError_t launch_block_extract(const float* Wd, float* W, int64_t d_in, int64_t d_out, int64_t G, bool accumulate,
                                hipStream_t st);
size_t quad_workspace_bytes(int64_t L, int64_t D);
size_t fft_next_pow2(int64_t L);
const char* fft_workspace_bytes(int64_t B, int64_t L, int64_t D, size_t* bytes);
const char* launch_fft_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                 const float* gamma, const float* omega, const float* amp, const float* phase,
                                 void* ws, hipStream_t st);
hipError_t launch_quad_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                 const float* gamma, const float* omega, const float* amp, const float* phase,
                                 float* K, hipStream_t st);
hipError_t launch_params_map(const float* tg, const float* tw, int64_t n, float alpha_min, float* gamma,
                             float* omega, hipStream_t st);
hipError_t launch_params_map_bwd(const float* tg, const float* tw, const float* dg, const float* dw, int64_t n,
                                 float* dtg, float* dtw, hipStream_t st);
hipError_t launch_diagnostics(const float* gamma, const float* omega, const float* amp, const float* phase, int64_t D,
                              int64_t M, int64_t T, float* hl, float* en, float* spec, hipStream_t st);
hipError_t launch_params_init(int64_t D, int64_t M, double hl_min, double hl_max, double per_min, double per_max,
                              double alpha_min, float* tg, float* tw, hipStream_t st);
hipError_t launch_decode_consts(int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                                const float* phase, float* tab, hipStream_t st);
template <typename TX, typename TY>
hipError_t launch_decode_tab(int64_t B, int64_t D, int64_t M, const void* x, void* y, const float* tab,
                             float* state, hipStream_t st);
template <typename TX, typename TY>
hipError_t launch_decode_steps(int64_t B, int64_t N, int64_t D, int64_t M, const void* x, void* y,
                               const float* gamma, const float* omega, const float* amp,
                               const float* phase, float* state, hipStream_t st);

// Segments per row of the backward for a device of num_cus compute units.
int bwd_segments(int64_t nchains, int64_t P, int num_cus);
// Channels per block of the backward.
inline int bwd_block_channels(int elem_bytes) { return 64 / elem_bytes; }

template <typename TX>
hipError_t launch_bwd(const BwdArgs& a, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

hipError_t launch_bwd_reduce(const Geometry& g, int nseg, const float* part, const float4* q0,
                             const ModeCarry* cc, const float* h0, float* dgamma, float* domega,
                             float* damp, float* dphase, float* dh0, hipStream_t st);

template <typename T>
hipError_t launch_epi_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H,
                          int dh, int K, const float* Ct, float lambda_c, const float* w, const float* s, int vec,
                          hipStream_t st);
// epilogue fused with the grouped output projection (one group per head)
size_t epi_proj_lds(int H, int dh, int K, int64_t d_out, bool bf16);
size_t epi_z_lds(int H, int dh, int K, bool bf16);
template <typename T>
hipError_t launch_epi_z_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H,
                            int K, const float* Ct, float lambda_c, const float* w, const float* s, int num_cus,
                            hipStream_t st);
template <typename T>
hipError_t launch_epi_proj_fwd(const void* y, const void* gate, const void* v, const void* Wo, void* out, void* z, int64_t B,
                               int64_t L, int H, int K, int64_t d_out, const float* Ct, float lambda_c,
                               const float* w, const float* s, int num_cus, hipStream_t st);
template <typename T>
hipError_t launch_epi_bwd(const void* y, const void* gate, const void* v, const void* dz, void* dy, void* dgate,
                          void* dv, int64_t B, int64_t L, int H, int dh, int K, const float* Ct, float lambda_c,
                          const float* w, const float* s, float* dCt, float* dlambda_c, float* dw, float* ds,
                          float* part, int vec, hipStream_t st);

}  // namespace res
