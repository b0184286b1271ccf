/*
 * mbscan.h -- C ABI of the MI355X (gfx950) selective-scan library libmbscan.so.
 *
 * The operation is the selective state-space scan that every MambaByte layer
 * runs over its byte sequence (MambaByte, Section 2, eq. (2), with the
 * discretisation of Appendix D and the output and gating rows of Table 8):
 *
 *   dlt_t  = softplus(delta_t + dt_bias)          (eq. (3); or delta_t + dt_bias when delta_softplus == 0)
 *   h_t[n] = exp(dlt_t A[n]) h_{t-1}[n] + dlt_t B_t[n] u_t    (ZOH on A, simplified Euler on B)
 *   y_t    = (sum_n C_t[n] h_t[n] + Dskip u_t) * z_t sigmoid(z_t)
 *
 * for every (batch b, channel d) row independently, starting from a carried
 * state h0 and optionally returning the final state: the resume capability
 * that speculative decoding needs to verify a drafted byte chunk from the
 * cached state and continue from it (Section 3 "Speculative decoding through
 * subword drafting"; Appendix F, Algorithm 1).  mb_scan_step is the
 * one-byte recurrent update used during generation (Section 2: the recurrence
 * is run directly at inference).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - All tensor pointers are DEVICE pointers (memory allocated with hipMalloc or
 *   by a framework on the GPU that is current for the calling thread), dense
 *   and row-major in the layouts stated below.  The caller owns every buffer;
 *   the library keeps no pointer after the call returns.
 * - Work is enqueued on `stream` (a hipStream_t; NULL means the default
 *   stream) and the call returns without waiting.  Argument errors are found
 *   on the host before anything is enqueued and return a negative mb_status;
 *   a launch failure returns MB_ERR_HIP.  Faults during execution surface at
 *   the caller's next synchronisation.  The library never prints or aborts.
 * - Element types: "act" tensors (u, delta, z, B, C and their step
 *   counterparts) share one type, in_dtype: MB_F32 (IEEE float) or MB_BF16
 *   (bfloat16).  A, Dskip, dt_bias, h0, h_last and the step state h are
 *   always float.  The output y has type out_dtype.  All arithmetic is fp32.
 * - Alignment: every pointer must be aligned to its element size.
 * - Sizes: batch, dim, seqlen >= 0 (an empty problem is valid and enqueues
 *   nothing, except that seqlen == 0 still writes h_last = h0, or zeros);
 *   dstate must be 16 (the n_state of every MambaByte model, Table 9), 8, 4,
 *   2 or 1.  Every element count an entry point derives from its sizes
 *   (batch * dim * seqlen, batch * dstate * seqlen, batch * dim * dstate and,
 *   with recorded positions, npos * batch * dim * dstate) must stay below
 *   2^56; a larger one returns MB_ERR_SHAPE.
 */
#ifndef MBSCAN_H
#define MBSCAN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MB_ABI_VERSION 6

typedef enum {
    MB_F32 = 0,
    MB_BF16 = 1
} mb_dtype;

typedef enum {
    MB_OK = 0,
    MB_ERR_NULL = -1,        /* a required pointer is NULL */
    MB_ERR_SHAPE = -2,       /* a size is negative or too large */
    MB_ERR_DTYPE = -3,       /* in_dtype or out_dtype is not an mb_dtype */
    MB_ERR_ALIGN = -4,       /* a pointer is not aligned to its element size */
    MB_ERR_UNSUPPORTED = -5, /* dstate not in {1, 2, 4, 8, 16}, a convolution width outside
                                1 .. 4, or a reserved field is set */
    MB_ERR_HIP = -6,         /* the HIP runtime reported an error when launching */
    MB_ERR_ALIAS = -7        /* an output overlaps an input it may not overlap */
} mb_status;

/* Problem description of mb_scan_fwd. */
typedef struct {
    int64_t batch;          /* B: independent sequences */
    int64_t dim;            /* D: channels (e * d in the paper's notation) */
    int64_t seqlen;         /* L: bytes in the sequence */
    int64_t dstate;         /* N: SSM state size per channel (n_state) */
    int32_t in_dtype;       /* mb_dtype of u, delta, z, Bmat, Cmat */
    int32_t out_dtype;      /* mb_dtype of y */
    int32_t delta_softplus; /* nonzero: dlt = softplus(delta + dt_bias); zero: dlt = delta + dt_bias */
    int32_t reserved;       /* must be 0 */
} mb_scan_desc;

/*
 * Forward selective scan over a whole sequence (Section 2, eq. (2); the
 * parallel-scan path of Section 2 "Implementation" that also verifies drafted
 * bytes in Algorithm 1).
 *
 *   u, delta     act   (B, D, L)  input x and the raw timestep, time contiguous
 *   A            float (D, N)     diagonal of A per channel (normally negative)
 *   Bmat, Cmat   act   (B, N, L)  input and output projections, shared by all
 *                                 channels of a batch element, time contiguous
 *   Dskip        float (D)        skip weight; NULL means 0
 *   dt_bias      float (D)        added to delta before softplus; NULL means 0
 *   z            act   (B, D, L)  gate input; NULL means no gate (y = C h + D u)
 *   h0           float (B, D, N)  initial state; NULL means zeros
 *   y            out   (B, D, L)  output; must not overlap any input
 *   h_last       float (B, D, N)  state after the last byte; NULL means not
 *                                 written.  It may be the same buffer as h0
 *                                 (each row reads its h0 before writing), but
 *                                 must not partially overlap it or any other
 *                                 argument.
 */
int mb_scan_fwd(const mb_scan_desc *desc,
                const void *u, const void *delta, const float *A,
                const void *Bmat, const void *Cmat,
                const float *Dskip, const float *dt_bias, const void *z,
                const float *h0, void *y, float *h_last, void *stream);

/*
 * mb_scan_fwd for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  The
 * arguments, the results (the same bits as mb_scan_fwd's) and the errors are
 * those of mb_scan_fwd; the call itself allocates nothing.
 *
 * Where mb_scan_fwd cuts a sequence into time segments (few rows, long
 * sequences) it allocates a carry buffer on the stream: one plane of
 * batch x dim x 128 bytes per pre-pass piece (1 or 2 per segment but the last)
 * and one for h0.  This entry point keeps that carry in a static device array of
 * 8 MiB instead: each GPU the library runs on holds its own copy until the
 * process ends.  A problem whose carry would exceed it returns MB_ERR_SHAPE
 * (on a 256-CU MI355X the forward's segment choice stays below 8 MiB: 7.3 MiB
 * for batch 1, dim 4608, L 65536).  The array keeps the last call's contents; nothing in it needs to
 * start at zero (the segment pre-pass writes every carry entry before the scan
 * reads it).  Every call on one GPU shares that GPU's array, so calls that may
 * overlap in time on one GPU (other streams, other threads) race: serialise
 * them, or use mb_scan_fwd.
 */
int mb_scan_fwd_noalloc(const mb_scan_desc *desc,
                        const void *u, const void *delta, const float *A,
                        const void *Bmat, const void *Cmat,
                        const float *Dskip, const float *dt_bias, const void *z,
                        const float *h0, void *y, float *h_last, void *stream);

/*
 * mb_scan_fwd that also records the state at requested positions.  The
 * verifier of Algorithm 1 (Appendix F) scans the drafted bytes in parallel,
 * finds the bifurcation position c and continues byte by byte from h_c; the
 * resumable scan of Section 3 ("Speculative decoding through subword
 * drafting") restarts from that state instead of from the first byte.
 *
 *   pos    int32 (npos, B)        pos[k * B + b] is the k-th requested
 *                                 position of batch element b: a timestep
 *                                 0 <= p < L, or -1 for the state before the
 *                                 first byte.  Positions need not be sorted or
 *                                 distinct.  Device memory, read only.
 *   npos   >= 0                   0 disables recording (pos and h_pos are then
 *                                 ignored and may be NULL).
 *   h_pos  float (npos, B, D, N)  h_pos[k][b][d][n] = h_p[n] of row (b, d)
 *                                 after timestep p = pos[k * B + b] (h0, or
 *                                 zeros, for p = -1).  A position outside
 *                                 [-1, L-1] is not an error: its slot is
 *                                 filled with NaN.  h_pos[k] has the layout of
 *                                 h0, so it can be passed back as h0 to resume
 *                                 every row of the batch from its k-th
 *                                 position.  h_pos must not overlap any other
 *                                 argument; pos must not overlap y or h_last.
 *
 * Every other argument is as for mb_scan_fwd, and y and h_last are the same
 * bits as mb_scan_fwd's.  A recorded state equals the state the scan carries
 * at that timestep bit for bit.
 */
int mb_scan_fwd_states(const mb_scan_desc *desc,
                       const void *u, const void *delta, const float *A,
                       const void *Bmat, const void *Cmat,
                       const float *Dskip, const float *dt_bias, const void *z,
                       const float *h0, void *y, float *h_last,
                       const int32_t *pos, int64_t npos, float *h_pos, void *stream);

/*
 * mb_scan_fwd that also stores the checkpoints mb_scan_bwd recomputes its
 * chunks from: the training forward (Section 4, Appendix C), whose backward
 * then skips its own forward pass over the sequence.
 *
 *   ck     float (L/16, B, D, N)   ck[k][b][d][n] = h_{16k-1}[n] of row (b, d),
 *                                  the state before timestep 16k (h0, or zeros,
 *                                  for k = 0).  Required; must not overlap any
 *                                  other argument; 8-byte aligned.
 *
 * Every other argument is as for mb_scan_fwd, and y and h_last are the same
 * bits as mb_scan_fwd's.  Supported: dstate 16, L a multiple of 16 below 2^25
 * (MB_ERR_UNSUPPORTED otherwise), u, delta, z, Bmat, Cmat and y 16-byte
 * aligned (MB_ERR_ALIGN otherwise).
 */
int mb_scan_fwd_ckpt(const mb_scan_desc *desc,
                     const void *u, const void *delta, const float *A,
                     const void *Bmat, const void *Cmat,
                     const float *Dskip, const float *dt_bias, const void *z,
                     const float *h0, void *y, float *h_last, float *ck, void *stream);

/*
 * One recurrent step per row, the state updated in place (Section 2:
 * generation runs the recurrence directly; Algorithm 1's byte-level
 * correction loop).  Identical to mb_scan_fwd with L = 1, h0 = h_last = h.
 *
 *   u_t, delta_t   act   (B, D)     this byte's input and raw timestep
 *   A              float (D, N)
 *   B_t, C_t       act   (B, N)
 *   Dskip, dt_bias float (D)        NULL means 0
 *   z_t            act   (B, D)     NULL means no gate
 *   h              float (B, D, N)  state, read then overwritten; required
 *   y_t            out   (B, D)     output; must not overlap any input or h
 *
 * dim must stay below 2^36 (the launch covers 64 channels per workgroup along
 * one grid dimension); a larger one returns MB_ERR_SHAPE.
 */
int mb_scan_step(int64_t batch, int64_t dim, int64_t dstate,
                 int32_t in_dtype, int32_t out_dtype, int32_t delta_softplus,
                 const void *u_t, const void *delta_t, const float *A,
                 const void *B_t, const void *C_t,
                 const float *Dskip, const float *dt_bias, const void *z_t,
                 float *h, void *y_t, void *stream);

/*
 * The backward of mb_scan_fwd (training at the 8,192-byte context: Section 4,
 * Appendix C): the gradients of sum(dy * y) + sum(dh_last * h_last) with
 * respect to every input of the scan, by reverse-mode differentiation of eq. (2)
 * with the discretisation of Appendix D and Table 8's output and gating.
 *
 *   desc, u, delta, A, Bmat, Cmat, Dskip, dt_bias, z, h0   as for mb_scan_fwd
 *   dy        out-dtype (B, D, L)   gradient with respect to y (desc->out_dtype)
 *   dh_last   float (B, D, N)       gradient with respect to h_last; NULL means 0
 *   ck        float (L/16, B, D, N) checkpoints written by mb_scan_fwd_ckpt for
 *                                   the same inputs, read only; NULL: the call
 *                                   computes them itself (one more forward pass)
 *   du, ddelta, dz   out-dtype (B, D, L)   dz is required when z is given
 *   dA        float (D, N)          summed over batch and time
 *   dB, dC    float (B, N, L)       summed over the channels of each batch element
 *   dDskip, ddt_bias float (D)      required when Dskip / dt_bias are given
 *   dh0       float (B, D, N)       NULL means not written
 * Outputs are overwritten (not accumulated) and must not overlap any other
 * argument; with no row (batch 0) dA, dDskip and ddt_bias are set to zero.
 * Supported: dstate 16, L a multiple of 16 below 2^25, every activation
 * pointer 16-byte aligned and every float pointer 8-byte aligned
 * (MB_ERR_UNSUPPORTED / MB_ERR_ALIGN otherwise).  Results are deterministic.  The call allocates a
 * stream-ordered workspace (hipMallocAsync): state checkpoints every 16 bytes
 * (L/16 x B x D x 16 floats, only when ck is NULL) and per-8-channel dB/dC
 * partials (B x L x D/8 x 64 bytes), freed on the same stream.
 */
int mb_scan_bwd(const mb_scan_desc *desc,
                const void *u, const void *delta, const float *A,
                const void *Bmat, const void *Cmat,
                const float *Dskip, const float *dt_bias, const void *z,
                const float *h0, const void *dy, const float *dh_last, const float *ck,
                void *du, void *ddelta, void *dz, float *dA, float *dB, float *dC,
                float *dDskip, float *ddt_bias, float *dh0, void *stream);

/*
 * The causal depthwise convolution upstream of the scan.  In the Mamba block
 * the x branch is convolved per channel over time with a short kernel and a
 * bias, then passed through the Swish activation, and the result is the scan's
 * input u (Table 8, "Pre-SSM 1D convolution"; Fig. 5, right; kernel size
 * k = 4 in every MambaByte model, Table 9):
 *
 *   pre_t = bias[d] + sum_{i < k} w[d][i] x_{t-(k-1)+i}
 *   y_t   = pre_t * sigmoid(pre_t)     (apply_silu != 0), else pre_t
 *
 * The k - 1 inputs before the first byte come from a carried state, so that a
 * sequence continues exactly where the previous call stopped, and the call
 * returns the last k - 1 inputs as the next state (the convolution's part of
 * the resume that Algorithm 1 relies on).  Arithmetic is fp32.
 */
typedef struct {
    int64_t batch;          /* B */
    int64_t dim;            /* D: channels (e * d) */
    int64_t seqlen;         /* L */
    int32_t width;          /* k: taps per channel, 1 .. 4 */
    int32_t in_dtype;       /* mb_dtype of x */
    int32_t out_dtype;      /* mb_dtype of y */
    int32_t apply_silu;     /* nonzero: Swish after the convolution */
    int32_t reserved;       /* must be 0 */
    int32_t reserved2;      /* must be 0 */
} mb_conv_desc;

/*
 *   x          act   (B, D, L)    input, time contiguous
 *   w          float (D, k)       taps; w[d][k-1] multiplies the current byte
 *   bias       float (D)          NULL means 0
 *   state_in   float (B, D, k-1)  the k-1 inputs before x, oldest first; NULL
 *                                 means zeros (the start of a sequence)
 *   y          out   (B, D, L)    output; must not overlap any other argument
 *   state_out  float (B, D, k-1)  the last k-1 inputs (of state_in followed by
 *                                 x); NULL means not written.  It must not
 *                                 overlap any other argument, state_in
 *                                 included: alternate two buffers to chain
 *                                 calls.  With L = 0 it receives state_in.
 * Errors as for mb_scan_fwd; a width outside 1 .. 4 or a nonzero reserved
 * field is MB_ERR_UNSUPPORTED.
 */
int mb_conv1d_fwd(const mb_conv_desc *desc, const void *x, const float *w, const float *bias,
                  const float *state_in, void *y, float *state_out, void *stream);

/*
 * One byte per row, the convolution state updated in place (generation, and
 * Algorithm 1's byte-level correction loop).  Identical to mb_conv1d_fwd with
 * L = 1, state_in = the old state and state_out = the new one.
 *
 *   x_t    act   (B, D)        this byte's input
 *   w      float (D, k), bias float (D) (NULL means 0)
 *   state  float (B, D, k-1)   read then overwritten; required when k > 1
 *   y_t    out   (B, D)        must not overlap any other argument
 */
int mb_conv1d_step(int64_t batch, int64_t dim, int32_t width, int32_t in_dtype, int32_t out_dtype,
                   int32_t apply_silu, const void *x_t, const float *w, const float *bias,
                   float *state, void *y_t, void *stream);

/*
 * The top-beta check that ends a speculative verification (Section 3,
 * "Speculative decoding through subword drafting"; Appendix F, Algorithm 1;
 * beta = 3 in Table 6).  For drafted byte i of batch element b:
 *
 *   rank   = 1 + the number of candidates y with logits[b][i][y] > logits[b][i][x],
 *            x = draft[b][i]; vocab + 1 when x is outside [0, vocab) or its logit
 *            is NaN (such a byte is always rejected).  Ties do not count against x.
 *            Logits rank exactly like probabilities (a softmax is monotone).
 *   accepted[b] = the number of leading drafted bytes whose rank is <= beta, i.e.
 *            the bifurcation position c: bytes 1..c verified, byte c+1 not.
 *   last_pos[b] = accepted[b] - 1, the 0-based timestep of the last accepted byte
 *            in the verified chunk (-1: none), which can be passed on device, as
 *            pos, to mb_scan_fwd_states to recover the state there.
 *
 *   logits    act   (batch, ndraft, vocab)  next-byte scores; logits[b][i] scores
 *                                            drafted byte i
 *   draft     int32 (batch, ndraft)          the drafted bytes
 *   beta      any int32 (<= 0 accepts nothing)
 *   ranks     int32 (batch, ndraft)          output; NULL means not written
 *   accepted  int32 (batch)                  output; required
 *   last_pos  int32 (batch)                  output; NULL means not written
 * Outputs must not overlap each other or the inputs.  vocab >= 1, ndraft and
 * vocab below 2^31.
 */
int mb_verify_rank(int64_t batch, int64_t ndraft, int64_t vocab, int32_t logit_dtype, int32_t beta,
                   const void *logits, const int32_t *draft, int32_t *ranks, int32_t *accepted,
                   int32_t *last_pos, void *stream);

/* Static, NUL-terminated description of a status code (never NULL). */
const char *mb_status_string(int status);

/* MB_ABI_VERSION of the built library. */
int mb_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MBSCAN_H */
