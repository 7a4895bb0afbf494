/*
 * resonator.h -- C ABI of the MI355X (gfx950) causal resonant field mixing library.
 *
 * The operator is ResonatorLM's replacement for self-attention (arXiv 2607.05583,
 * Sec. 3).  Per channel d the drive x[b, t, d] is mixed causally through a bank of
 * M damped resonators:
 *
 *   K_d[tau] = sum_m a[d,m] exp(-gamma[d,m] tau) cos(omega[d,m] tau + phi[d,m])   (Sec. 3.1, kernel eq.)
 *   y[b,t,d] = sum_{s<=t} K_d[t-s] x[b,s,d]  +  Re sum_m c[d,m] lambda[d,m]^(t+1) h0[b,d,m]
 *                                                                                 (Sec. 3.2, causal conv eq.)
 * equivalently the complex diagonal recurrence (Sec. 3.3)
 *   h_t = lambda h_{t-1} + x_t,  h_{-1} = h0,  y_t = Re sum_m c h_t,
 *   lambda = exp(-gamma) (cos omega + i sin omega),  c = a (cos phi + i sin phi).
 * The readout phase sign follows the kernel of Sec. 3.1 (the decode equation of
 * Sec. 3.3 prints e^{-i phi}; with it decode would not reproduce the kernel).
 *
 * Conventions shared by every entry point
 *   - All pointers are DEVICE pointers unless stated otherwise; the caller owns
 *     every buffer (inputs, outputs, workspace).  Apart from two thread-local
 *     items (the last error text and the armed measurement hook) the library
 *     keeps no state between calls and is safe to call from several host threads.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL = the default stream).  It returns once the kernels are enqueued.
 *   - Activations x, y, dy, dx: row-major [B][L][D] (channels fastest), element
 *     type given by a res_dtype_t.  bfloat16 is stored as its 16-bit pattern and
 *     rounded to nearest even on output.  Arithmetic is float32 (MFMA with fp32
 *     accumulation; bf16 MFMA operands when activations are bf16), with the
 *     parameter-derived constants computed in float64 from exact integer lags.
 *   - Parameters gamma, omega, amp, phase: float32 [D][M], row-major (m fastest).
 *     gamma >= 0 is a precondition (not checked on the device); any finite omega,
 *     amp, phase is accepted as given (no clamping).
 *   - States (h0, h_out, state): float32 [B][D][M][2] = (re, im) interleaved.
 *   - Sizes are int64; B, D >= 1, L >= 1 (L_prompt >= 0 for state_init),
 *     1 <= M <= RES_M_MAX.
 *   - Pointer alignment: float32 tensors 4 bytes, bf16 tensors 2 bytes, the
 *     workspace 256 bytes.
 *   - Errors: a non-OK status means nothing was launched and no output was
 *     touched; resonator_last_error() then returns a description (thread-local).
 *     RES_ERR_HIP reports a failed launch; faults inside kernels surface at the
 *     caller's next synchronisation.  No C++ exception crosses the ABI.
 */
#ifndef RESONATOR_H
#define RESONATOR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { RES_F32 = 0, RES_BF16 = 1 } res_dtype_t;

enum {
  RES_OK = 0,
  RES_ERR_INVALID_ARG = 1,   /* null pointer, bad size, aliasing, bad op code   */
  RES_ERR_UNSUPPORTED = 2,   /* dtype pair or M outside what the kernels support */
  RES_ERR_MISALIGNED = 3,    /* pointer not aligned as stated above              */
  RES_ERR_WORKSPACE = 4,     /* workspace null or smaller than required          */
  RES_ERR_HIP = 5            /* HIP runtime error when launching                 */
};

enum { RES_OP_FWD = 0, RES_OP_BWD = 1, RES_OP_STATE_INIT = 2 };

#define RES_M_MAX 16

/* Library ABI version (major * 100 + minor). */
int resonator_version(void);

/*
 * Bytes of device workspace that op (RES_OP_*) needs for activations of type
 * act_dt at sizes (B, L, D, M).  Returns 0 for invalid arguments.  The workspace
 * holds parameter tables, per-tile chunk states, carries and (for bwd) per-tile
 * partial sums.
 *   - RES_OP_FWD: the workspace must be zero-filled before its first forward call;
 *     every forward call leaves it ready for the next one (any sizes whose need
 *     it covers).  Its first 4 bytes are the forward status word (see
 *     resonator_fwd_status).  Forward calls that share a workspace must not
 *     overlap in time.
 *   - RES_OP_BWD, RES_OP_STATE_INIT: contents need not be initialised and are
 *     clobbered.
 */
size_t resonator_workspace_bytes(int op, res_dtype_t act_dt, int64_t B, int64_t L, int64_t D,
                                 int64_t M);

/*
 * Forward mixing (Sec. 3.1 kernel, Sec. 3.2 causal convolution).
 *   x      [B][L][D] of x_dt            drive
 *   y      [B][L][D] of y_dt            output; must not overlap x
 *   gamma, omega, amp, phase [D][M]     float32 resonator parameters
 *   h0     [B][D][M][2] or NULL         state before t = 0 (NULL = zero)
 *   h_out  [B][D][M][2] or NULL         terminal state h_{L-1} (may alias h0)
 *   ws     workspace of resonator_workspace_bytes(RES_OP_FWD, x_dt, B, L, D, M)
 * Supported (x_dt, y_dt): (F32, F32), (BF16, BF16), (BF16, F32).
 */
int resonator_mix_fwd(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B,
                      int64_t L, int64_t D, int64_t M, const float* gamma, const float* omega,
                      const float* amp, const float* phase, const float* h0, float* h_out,
                      void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of resonator_mix_fwd for the loss sum(dy * y) (gradients derived from
 * the Sec. 3.1 kernel; the paper trains through autograd and prints none).
 *   x, dy  [B][L][D] of act_dt          forward drive and upstream gradient
 *   dx     [B][L][D] of act_dt          gradient w.r.t. x (overwritten)
 *   h0     [B][D][M][2] or NULL         the forward's initial state (NULL = zero)
 *   dgamma, domega, damp, dphase [D][M] float32, overwritten (not accumulated)
 *   dh0    [B][D][M][2] or NULL         gradient w.r.t. h0 (overwritten)
 *   ws     workspace of resonator_workspace_bytes(RES_OP_BWD, act_dt, B, L, D, M)
 * act_dt is F32 or BF16.  dx must not overlap x or dy.  Parameter gradients are
 * reduced in a fixed order (float64), so they are bitwise reproducible.
 */
int resonator_mix_bwd(const void* x, const void* dy, res_dtype_t act_dt, void* dx, int64_t B,
                      int64_t L, int64_t D, int64_t M, const float* gamma, const float* omega,
                      const float* amp, const float* phase, const float* h0, float* dgamma,
                      float* domega, float* damp, float* dphase, float* dh0, void* ws,
                      size_t ws_bytes, void* stream);

/*
 * Forward status word (the first 4 bytes of a forward workspace), an OR over the
 * forward calls made with ws since it was last cleared:
 *   bit 0  a bounded wait for another work-group's published state gave up (the
 *          outputs of that call are wrong);
 *   bit 1  the workspace counters were not in their initial state when a call
 *          started (workspace not zero-filled before first use, or used by
 *          overlapping calls): that call computed nothing and left y untouched.
 * Neither happens with a zero-filled workspace used by one call at a time.  This
 * call enqueues a copy of the word into *status (host memory) and a clear of the
 * word on stream, then synchronises the stream.  Returns RES_OK, or
 * RES_ERR_INVALID_ARG / RES_ERR_MISALIGNED / RES_ERR_HIP.
 */
int resonator_fwd_status(void* ws, uint32_t* status, void* stream);
/* The same for the static scratch of resonator_mix_fwd_noalloc on the current device. */
int resonator_fwd_status_noalloc(uint32_t* status, void* stream);

/*
 * Allocation-free forward, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Computes exactly what resonator_mix_fwd computes, with the same
 * arguments except the workspace: the library uses a static device array of
 * RES_NOALLOC_SCRATCH_BYTES bytes instead, one per GPU, held until the process
 * ends.  The call allocates nothing (no hipMalloc, no allocating library call).
 *   - stream must belong to the calling thread's current device (NULL = that
 *     device's default stream); else RES_ERR_INVALID_ARG.
 *   - Sizes whose resonator_workspace_bytes(RES_OP_FWD, ...) exceed
 *     RES_NOALLOC_SCRATCH_BYTES return RES_ERR_WORKSPACE with nothing launched.
 *   - All calls on one GPU share its scratch: calls that overlap in time on one
 *     GPU (concurrent streams, several host threads) race and give wrong results;
 *     calls ordered on one stream are safe.
 *   - The first call on a device looks up the scratch's device address (not
 *     inside a graph capture: make one call before capturing).
 * Other arguments, dtypes, alignment and errors as resonator_mix_fwd.
 */
#define RES_NOALLOC_SCRATCH_BYTES (32u << 20)
int resonator_mix_fwd_noalloc(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B, int64_t L,
                              int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                              const float* phase, const float* h0, float* h_out, void* stream);
/* RES_NOALLOC_SCRATCH_BYTES, the largest workspace resonator_mix_fwd_noalloc can serve. */
size_t resonator_mix_fwd_noalloc_max_bytes(void);

/*
 * Prompt state for decoding (Sec. 3.2, cache construction): the terminal state
 * state[b,d,m] = sum_s lambda^(L-1-s) x[b,s,d], each drive scaled by the pole
 * raised to its age (newest drive weight 1), from a zero initial state.
 *   x_prompt  [B][L_prompt][D] of x_dt, may be NULL when L_prompt == 0
 *   state_out [B][D][M][2] float32       written
 *   ws        workspace of resonator_workspace_bytes(RES_OP_STATE_INIT, x_dt, B, L_prompt, D, M)
 *             (may be NULL / 0 bytes when L_prompt == 0)
 */
int resonator_state_init(const void* x_prompt, res_dtype_t x_dt, int64_t B, int64_t L_prompt,
                         int64_t D, int64_t M, const float* gamma, const float* omega,
                         const float* amp, const float* phase, float* state_out, void* ws,
                         size_t ws_bytes, void* stream);

/*
 * One recurrent decode step for every (b, d) (Sec. 3.3):
 *   state <- lambda state + x_t;   y_t = Re sum_m c state.
 *   x_t    [B][D] of x_dt;  y_t [B][D] of y_dt (not overlapping x_t or state)
 *   state  [B][D][M][2] float32, read and updated in place
 * lambda is applied as a float32 hi + lo pair computed in float64, so long runs
 * do not accumulate the phase error of a single rounded pole.
 * Supported (x_dt, y_dt) as for resonator_mix_fwd.  Needs no workspace.
 */
int resonator_decode_step(const void* x_t, res_dtype_t x_dt, void* y_t, res_dtype_t y_dt,
                          int64_t B, int64_t D, int64_t M, const float* gamma, const float* omega,
                          const float* amp, const float* phase, float* state, void* stream);

/*
 * Decode from a constants table (Sec. 3.3), for token-by-token loops:
 * resonator_decode_constants evaluates, once, the per-(channel, mode) constants
 * that resonator_decode_step evaluates on every call,
 *   tab [D][M][6] float32 = (Re, Im) of lambda's float32 pair hi and lo, and of c,
 * and resonator_decode_step_tab runs one step from it.  The step's arithmetic and
 * its order are those of resonator_decode_step, so the results are bitwise the
 * same.  tab: device memory of D*M*24 bytes, 16-byte aligned for the fast path,
 * owned by the caller; it stays valid until the parameters change.  Other
 * arguments, layouts and errors as for resonator_decode_step.  Needs no
 * workspace.
 */
int resonator_decode_constants(int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                               const float* phase, float* tab, void* stream);
int resonator_decode_step_tab(const void* x_t, res_dtype_t x_dt, void* y_t, res_dtype_t y_dt, int64_t B,
                              int64_t D, int64_t M, const float* tab, float* state, void* stream);

/*
 * N decode steps in one launch, for drives known in advance (a prompt chunk,
 * drafted tokens to verify) (Sec. 3.3):
 *   for n = 0 .. N-1:  state <- lambda state + x[:, n];  y[:, n] = Re sum_m c state.
 *   x      [B][N][D] of x_dt;  y [B][N][D] of y_dt (not overlapping x or state)
 *   state  [B][D][M][2] float32, read once and written once, in place
 * Each step uses the constants, arithmetic and order of resonator_decode_step,
 * so the results are bitwise those of N calls of it.  Supported (x_dt, y_dt) as
 * for resonator_mix_fwd.  N >= 1, B <= 262140.  Needs no workspace.
 */
int resonator_decode_steps(const void* x, res_dtype_t x_dt, void* y, res_dtype_t y_dt, int64_t B, int64_t N,
                           int64_t D, int64_t M, const float* gamma, const float* omega, const float* amp,
                           const float* phase, float* state, void* stream);

/*
 * Grouped linear projection (Sec. 3.1 drive and gate projection, Sec. 3.4
 * output projection): a block-diagonal weight of G groups,
 *   y[n, g dq + j] = sum_i x[n, g di + i] W[g][i][j],   di = d_in / G, dq = d_out / G.
 *   x  [N][d_in], W [G][d_in/G][d_out/G], y [N][d_out], all of dtype dt (bf16 or
 *      f32), device memory, row-major; y must not overlap x or W
 * Float32 accumulation, on the given stream.  When d_in/G is a multiple of 32
 * (bf16) or 16 (f32), d_out/G a multiple of 16 and at most 128, a row of x at
 * most 1 KB, the weight at most 64 KB (32 KB with bf16 for
 * resonator_grouped_linear2) and x, W and y 16-byte aligned, it runs as the
 * library's own MFMA kernel (16 tokens per wave, weights staged in LDS; bf16
 * outputs rounded once); other shapes go to one rocBLAS strided-batched GEMM.
 * Calls from several host threads on one device must not overlap (they share
 * that device's rocBLAS handle).  N, d_in, d_out < 2^31.
 */
int resonator_grouped_linear(const void* x, const void* W, res_dtype_t dt, void* y, int64_t N, int64_t d_in,
                             int64_t d_out, int64_t G, void* stream);

/*
 * Two grouped projections of the same input (Sec. 3.1: the drive u and the gate
 * g are both projections of the block input), from one read of x:
 *   y0 = x W0,  y1 = x W1   (each as resonator_grouped_linear; W0 and W1 of
 *   the same shape [G][d_in/G][d_out/G]; y0 and y1 [N][d_out], overlapping
 *   neither each other, x, W0 nor W1).
 * Shapes the MFMA kernel does not take run as two library GEMMs.  Errors as
 * resonator_grouped_linear.
 */
int resonator_grouped_linear2(const void* x, const void* W0, const void* W1, res_dtype_t dt, void* y0, void* y1,
                              int64_t N, int64_t d_in, int64_t d_out, int64_t G, void* stream);

/*
 * Backward of resonator_grouped_linear (loss sum(dy * y)):
 *   data:    dx[n, g di + i] = sum_j dy[n, g dq + j] W[g][i][j]     (dx of dtype dt)
 *   weight:  dW[g][i][j]    = sum_n x[n, g di + i] dy[n, g dq + j]  (dW float32)
 * With accumulate != 0 the result is added to the output instead of replacing
 * it (gradients of several uses of one input or weight).  Same array
 * conventions as the forward; outputs must not overlap the inputs.
 */
int resonator_grouped_linear_bwd_data(const void* dy, const void* W, res_dtype_t dt, void* dx, int64_t N,
                                      int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* stream);
int resonator_grouped_linear_bwd_weight(const void* x, const void* dy, res_dtype_t dt, float* dW, int64_t N,
                                        int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* stream);

/*
 * Data gradient of n = 1..3 grouped projections of one input (Sec. 3.1: the
 * block input feeds both the drive and the gate projection, so its gradient is
 * the sum of theirs):
 *   dx[n, g di + i] (+)= sum_{k < n} sum_j dy[k][n, g dq + j] W[k][g][i][j]
 * dy and W are host arrays of n device pointers (dy[k] [N][d_out], W[k]
 * [G][d_in/G][d_out/G], all of dtype dt); the sum is formed in float32 and dx
 * (dtype dt) is written once.  With accumulate != 0 dx's present value is added
 * first.  When d_out/G is a multiple of 32 (bf16) or 16 (f32), d_in/G a multiple
 * of 16 and at most 128, d_out at most 256 elements (512 bytes of a row with
 * n = 1), the n weights at most 64 KB and every array 16-byte aligned, it runs as
 * the library's own MFMA kernel (the weights staged transposed in LDS); other
 * shapes go to n rocBLAS strided-batched GEMMs.  resonator_grouped_linear_bwd_data
 * is this call with n = 1.  dx must not overlap any dy[k] or W[k]; n outside
 * 1..3 is RES_ERR_INVALID_ARG.
 */
int resonator_grouped_linear_bwd_data_sum(int n, const void* const* dy, const void* const* W, res_dtype_t dt,
                                          void* dx, int64_t N, int64_t d_in, int64_t d_out, int64_t G,
                                          int accumulate, void* stream);

/*
 * Weight gradients of n = 1..3 grouped projections of one input x (Sec. 3.1:
 * the drive's gradient enters W_u twice, from the mixing and from the local
 * path, and the gate's enters W_g; Sec. 3.4: the output projection):
 *   dW_m[g][i][j] (+)= sum_{k < n, out[k] = m} sum_t x[t, g di + i] dy[k][t, g dq + j]
 * for m = 0 and, when some out[k] = 1, m = 1 (dW0, dW1 float32 [G][d_in/G][d_out/G]).
 * dy and out are host arrays of n entries (device pointers, weight indices 0 or
 * 1; at least one gradient goes to weight 0).  With bf16, d_in and d_out
 * multiples of 64 and at most 256, d_in/G and d_out/G multiples of 16, at most
 * 64 output blocks of 16 x 16 over both weights, and x and dy 16-byte aligned, it
 * runs as the library's own MFMA kernel: each work-group sums a token range
 * (32-token chunks staged in LDS and read down the columns) into partials in
 * ws, and a second kernel adds the partials in a fixed order, so the result is
 * deterministic.  Other shapes go to one rocBLAS strided-batched GEMM per
 * gradient and need no workspace.  ws: at least
 * resonator_grouped_linear_bwd_weight_sum_workspace_bytes(n, nout, N, d_in,
 * d_out, G, dt) bytes (nout = 2 when some out[k] = 1), 16-byte aligned, owned by
 * the caller, contents irrelevant; a smaller workspace where one is needed is
 * RES_ERR_INVALID_ARG.  The outputs must not overlap x, dy, ws or each other.
 */
size_t resonator_grouped_linear_bwd_weight_sum_workspace_bytes(int n, int nout, int64_t N, int64_t d_in,
                                                                int64_t d_out, int64_t G, res_dtype_t dt);
int resonator_grouped_linear_bwd_weight_sum(int n, const void* x, const void* const* dy, const int* out,
                                            res_dtype_t dt, float* dW0, float* dW1, int64_t N, int64_t d_in,
                                            int64_t d_out, int64_t G, int accumulate, void* ws, size_t ws_bytes,
                                            void* stream);

/*
 * Dense [d_in][d_out] copy of a grouped weight W [G][d_in/G][d_out/G], zero off
 * the diagonal blocks, so that resonator_grouped_linear with G = 1 on it gives
 * exactly the grouped product (the zero blocks add exact zeros) with the GEMM
 * library's efficient tile shapes.  Same dtype conventions; W_dense must not
 * overlap W; d_in d_out <= 2^31.
 */
int resonator_block_diag_weight(const void* W, res_dtype_t dt, int64_t d_in, int64_t d_out, int64_t G,
                                void* W_dense, void* stream);

/*
 * Grouped weight gradient with the contraction split (Sec. 3.1, 3.4
 * projections): the same result as resonator_grouped_linear_bwd_weight, for a
 * long contraction (N tokens) over small weights.  The N rows are cut into at
 * most 64 chunks (at least 256 rows each); one batched GEMM writes each chunk's
 * dense float32 product x_s^T dy_s [d_in][d_out] into the workspace, and a
 * second kernel sums the chunks' diagonal blocks in a fixed order into
 * dW [G][d_in/G][d_out/G] (added when accumulate != 0).  Deterministic.
 *   ws   resonator_grouped_linear_bwd_weight_split_workspace_bytes(N, d_in,
 *        d_out) bytes of device memory, 256-byte aligned, not overlapping the
 *        other arguments (0 from the size query means invalid sizes)
 * Other arguments, dtypes and errors as resonator_grouped_linear_bwd_weight;
 * d_in d_out <= 2^31.
 */
size_t resonator_grouped_linear_bwd_weight_split_workspace_bytes(int64_t N, int64_t d_in, int64_t d_out);
int resonator_grouped_linear_bwd_weight_split(const void* x, const void* dy, res_dtype_t dt, float* dW, int64_t N,
                                              int64_t d_in, int64_t d_out, int64_t G, int accumulate, void* ws,
                                              size_t ws_bytes, void* stream);

/*
 * The diagonal blocks of a dense float32 [d_in][d_out] matrix into a grouped
 * W [G][d_in/G][d_out/G] (W[g] = W_dense[g-th row block][g-th column block]),
 * added into W when accumulate != 0.  With the dense weight gradient from
 * resonator_grouped_linear_bwd_weight with G = 1, this gives the grouped weight
 * gradients (Sec. 3.1, 3.4 projections) from one efficient GEMM.  Device
 * memory, caller-owned, 4-byte aligned; W must not overlap W_dense;
 * d_in d_out <= 2^31.
 */
int resonator_block_diag_extract(const float* W_dense, int64_t d_in, int64_t d_out, int64_t G, float* W,
                                 int accumulate, void* stream);

/*
 * Quadratic causal reference mixer: the baseline of the kernel-tail benchmark
 * (Sec. 5.3, Table 5), not part of the mixing path.  Computes
 *   y[b,t,d] = sum_{s<=t} K_d[t-s] x[b,s,d],  K_d[tau] = sum_m a exp(-gamma tau) cos(omega tau + phi)
 * directly, O(L^2 D) float32 multiply-adds, with the taps tabulated per call in
 * float64 (rounded to float32) into the workspace.
 *   x, y   [B][L][D] float32 device memory (y must not overlap x or ws)
 *   ws     resonator_quadratic_reference_workspace_bytes(L, D) bytes, 4-byte aligned
 * B <= 65535, L D <= 2^31; otherwise as resonator_mix_fwd.
 */
size_t resonator_quadratic_reference_workspace_bytes(int64_t L, int64_t D);
int resonator_quadratic_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                                  const float* gamma, const float* omega, const float* amp, const float* phase,
                                  void* ws, size_t ws_bytes, void* stream);

/*
 * FFT causal convolution: the paper's own prefill evaluation of the mixing
 * (Sec. 3.2, the FFT form), kept as a baseline for the chunked scan, not part
 * of the mixing path.  Per channel d, with n the next power of two >= 2L,
 *   y[b,:,d] = IFFT( FFT(x[b,:,d] zero-padded to n) . FFT(K_d zero-padded to n) )[0:L]
 * in float32 through rocFFT (batched real transforms), with the taps K_d[tau],
 * tau < L, evaluated in float64 and rounded to float32.  Zero initial state.
 *   x, y   [B][L][D] float32 device memory (y must not overlap x or ws)
 *   ws     resonator_fft_reference_workspace_bytes(B, L, D) bytes, 256-byte
 *          aligned: the padded time-major signal [B D][n+2], the padded taps
 *          [D][n+2] and rocFFT's work area
 * Plans are created on first use per (device, n, batch) and kept for the
 * process; the workspace-size query creates them too (it returns 0 on error,
 * with the message in resonator_last_error).  B <= 65535, L <= 2^26.
 */
size_t resonator_fft_reference_workspace_bytes(int64_t B, int64_t L, int64_t D);
int resonator_fft_reference(const float* x, float* y, int64_t B, int64_t L, int64_t D, int64_t M,
                            const float* gamma, const float* omega, const float* amp, const float* phase, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * Constrained parameterization (Sec. 3.1, last paragraph): unconstrained
 * parameters are mapped into the valid ranges of the damping and frequency,
 *   gamma = alpha_min + softplus(theta_gamma)      (> alpha_min; the paper's floor is 1e-4)
 *   omega = pi * sigmoid(theta_omega)              (in (0, pi))
 * amplitude and phase are used as they are.  Arrays are float32 of n elements
 * (the [D][M] bank flattened), device memory, caller-owned; outputs must not
 * overlap each other.  n in [1, 2^31].
 */
int resonator_params_map(const float* theta_gamma, const float* theta_omega, int64_t n, float alpha_min,
                         float* gamma, float* omega, void* stream);

/*
 * Chain rule of resonator_params_map:
 *   dtheta_gamma = dgamma * sigmoid(theta_gamma)
 *   dtheta_omega = domega * pi * sigmoid(theta_omega) * (1 - sigmoid(theta_omega))
 * Same array conventions; the two outputs must not overlap.
 */
int resonator_params_map_bwd(const float* theta_gamma, const float* theta_omega, const float* dgamma,
                             const float* domega, int64_t n, float* dtheta_gamma, float* dtheta_omega,
                             void* stream);

/*
 * Initialization with log-spaced timescales (Sec. 3.1, last paragraph): writes
 * theta_gamma, theta_omega [D][M] whose mapped values have half-lives
 * ln 2 / gamma log-spaced from hl_min to hl_max and periods 2 pi / omega
 * log-spaced from per_max down to per_min, over the M modes of every channel
 * (over the D channels when M = 1, one mode per head as in the paper).  Needs
 * 0 < hl_min <= hl_max, 2 <= per_min <= per_max and ln 2 / hl_max > alpha_min.
 * The paper reports half-lives from about 2 to 2048 tokens.
 */
int resonator_params_init(int64_t D, int64_t M, double hl_min, double hl_max, double per_min, double per_max,
                          float alpha_min, float* theta_gamma, float* theta_omega, void* stream);

/*
 * Diagnostics of a mode bank (Sec. 3.5), float32 outputs, each nullable:
 *   half_life [D][M]   ln 2 / gamma;
 *   energy    [D][M][T] exp(-2 gamma t), t = 0 .. T-1 (state energy decay);
 *   spectrum  [T/2 + 1][D] |sum_{tau<T} K_d[tau] e^{-2 pi i k tau / T}|, the
 *             magnitude of the real DFT of the length-T impulse response
 *             K_d[tau] = Re sum_m c_m lambda_m^tau (Sec. 3.1), evaluated in
 *             closed form per mode in float64 (a geometric sum per bin).
 * gamma, omega, amp, phase [D][M] float32 device arrays (omega, amp and phase
 * may be null when spectrum is).  T >= 1 when energy or spectrum is asked for.
 * Outputs must not overlap the parameters or each other; invalid sizes or null
 * parameters are RES_ERR_INVALID_ARG.
 */
int resonator_diagnostics(const float* gamma, const float* omega, const float* amp, const float* phase, int64_t D,
                          int64_t M, int64_t T, float* half_life, float* energy, float* spectrum, void* stream);

/*
 * Mixer epilogue around the mixing output (Sec. 3.4, head coupling and local
 * lexical path; the gate of Sec. 3.1's last paragraph):
 *   C = I + (lambda_c / sqrt(H)) tanh(Ct)                          (coupling eq.)
 *   ybar[b,t,g*dh+j] = sum_h C[g][h] y[b,t,h*dh+j]                 (head mixing eq.)
 *   l[b,t,c] = sum_{k<K} w[c][k] v[b,t-k,c]  (zero before t = 0)   (causal depthwise conv)
 *   z = sigmoid(gate) * ybar + s * l                               (combine eq.)
 *   y, gate, v, z  [B][L][D] of act_dt, D = H * dh, channel c = h * dh + j
 *                  (v: the token stream the local path reads; may be NULL when K == 0)
 *   Ct [H][H], w [D][K], s [D]  float32 device arrays (w, s may be NULL when K == 0)
 *   lambda_c       coupling strength (host value); 0 gives uncoupled heads
 * 1 <= H <= 32, dh >= 1, 0 <= K <= 16 (K = 0: no local path).  z must not
 * overlap y, gate or v.  Needs no workspace.
 */
int resonator_epilogue_fwd(const void* y, const void* gate, const void* v, res_dtype_t act_dt, void* z,
                           int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K, const float* Ct,
                           float lambda_c, const float* w, const float* s, void* stream);

/* Workspace bytes of resonator_epilogue_bwd (0 for invalid sizes). */
size_t resonator_epilogue_workspace_bytes(int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K);

/*
 * The mixer epilogue fused with the grouped output projection (Sec. 3.4: the
 * combine equation, then the grouped output projection), one group per head:
 *   out[b, t, g dq + o] = sum_j z[b, t, g dh + j] Wo[g][j][o],   dq = d_out / H,
 *   z as resonator_epilogue_fwd (rounded to act_dt as it would store it).
 *   y, gate, v  [B][L][H dh] of act_dt; Wo [H][dh][d_out/H] of act_dt;
 *   out [B][L][d_out] of act_dt, overlapping none of the inputs; parameters as
 *   resonator_epilogue_fwd.
 * z stays in registers, so the call reads y, gate and v once and writes out once;
 * z (nullable, [B][L][H dh] of act_dt, 16-byte aligned, overlapping no other
 * argument) also receives it, bitwise resonator_epilogue_fwd's output, for a
 * backward that keeps the forward's intermediates.  The result is bitwise that
 * of resonator_epilogue_fwd followed by
 * resonator_grouped_linear on the MFMA kernel.  Takes H <= 8, dh = 32 (bf16) or
 * 16 (f32), K <= 4, d_out/H = 16 or 32, and y, gate, v, Wo and out 16-byte
 * aligned; other shapes return RES_ERR_UNSUPPORTED (run the two calls instead),
 * misaligned pointers RES_ERR_MISALIGNED.
 */
int resonator_epilogue_proj_fwd(const void* y, const void* gate, const void* v, res_dtype_t act_dt, const void* Wo,
                                void* out, void* z, int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K,
                                int64_t d_out, const float* Ct, float lambda_c, const float* w, const float* s,
                                void* stream);

/*
 * Backward of resonator_epilogue_fwd for the loss sum(dz * z):
 *   dz               [B][L][D] of act_dt
 *   dy, dgate, dv    [B][L][D] of act_dt, overwritten (dv may be NULL when K == 0);
 *                    none may overlap the inputs or each other
 *   dCt [H][H], dw [D][K], ds [D], dlambda_c [1]  float32 device arrays, overwritten
 *                    (dw, ds may be NULL when K == 0)
 *   ws               workspace of resonator_epilogue_workspace_bytes(B, L, H, dh, K)
 * The parameter gradients are reduced in a fixed order (per block of rows, then
 * over blocks in float64), so they are bitwise reproducible.
 */
int resonator_epilogue_bwd(const void* y, const void* gate, const void* v, const void* dz, res_dtype_t act_dt,
                           void* dy, void* dgate, void* dv, int64_t B, int64_t L, int64_t H, int64_t dh, int64_t K,
                           const float* Ct, float lambda_c, const float* w, const float* s, float* dCt,
                           float* dlambda_c, float* dw, float* ds, void* ws, size_t ws_bytes, void* stream);

/*
 * Measurement hook.  Arms a pair of HIP events (hipEvent_t passed as void*) on the
 * calling thread: the next resonator_mix_fwd or resonator_mix_bwd call on this
 * thread records start_event immediately before and stop_event immediately after
 * its dominant kernel (the one that reads the activations and writes the output),
 * on the call's stream; the hook then disarms itself.  Pass NULL, NULL to disarm.
 * The events belong to the caller.  Returns RES_OK, or RES_ERR_INVALID_ARG if
 * exactly one of the two is NULL.
 */
int resonator_set_kernel_timer(void* start_event, void* stop_event);

/* Text describing the last non-OK status returned on this thread. */
const char* resonator_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RESONATOR_H */
