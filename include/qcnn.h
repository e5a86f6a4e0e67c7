/*
 * qcnn.h -- C ABI of the product-quantized (PQ) layer forward on AMD MI355X
 * (gfx950).
 *
 * Method: J. Wu, C. Leng, Y. Wang, Q. Hu, J. Cheng, "Quantized Convolutional
 * Neural Networks for Mobile Devices", CVPR 2016 (arXiv 1512.06473).
 *
 * Notation (Sec. 2 and 3 of the paper): a layer has C_s input and C_t output
 * channels.  The C_s-dimensional input space is split evenly into M subspaces
 * of C'_s = C_s / M consecutive channels (Sec. 3.1; Sec. 3.2 splits a conv
 * kernel along its input channels).  Subspace m has a sub-codebook D^(m) of K
 * sub-codewords of length C'_s, and every weight sub-vector is stored as the
 * index of one sub-codeword: k_m(c_t) for a fully-connected layer (Eq. (5)),
 * k_m(c_t, p_k) for a conv kernel at offset p_k (Eq. (7)).
 *
 * Test phase (Sec. 3.1, the paragraph after Eq. (5); Sec. 3.2 after Eq. (7)):
 *   1. table:  L[m][k][p_s] = < D^(m)_k , S^(m)_{p_s} >  at each input position;
 *   2. gather: each response is the sum of M (conv: M d_k^2) table entries
 *      selected by the codes.
 *
 * Conventions shared by every entry point
 *   - All pointers are DEVICE pointers on the current HIP device (torch CUDA
 *     tensors on ROCm qualify), C-contiguous, fp32 unless noted.  The caller
 *     owns every buffer; the library never frees, retains or caches a caller
 *     pointer beyond the call.
 *   - Layouts: feature maps NCHW [N][C][H][W]; codebooks [M][K][C'_s] (row k
 *     of subspace m is D^(m)_k); conv codes uint8 [C_t][d_k][d_k][M] with
 *     codes[t][ky][kx][m] = k_m(c_t, (ky, kx)); FC codes uint8 [C_t][M] with
 *     codes[t][m] = k_m(c_t).
 *   - The conv pairing of input and kernel positions (Eq. (1)) is
 *     cross-correlation: input row  yo * stride - pad + ky, column
 *     xo * stride - pad + kx; positions in the zero padding contribute 0.
 *     H_o = floor((H + 2 pad - d_k) / stride) + 1, likewise W_o.
 *   - Optional bias [C_t] (NULL for none) is added after the sum, then ReLU if
 *     relu != 0.  Neither is part of Eq. (5)/(7); NULL/0 give exactly those.
 *   - Limits: 1 <= K <= 256 (codes are uint8), 1 <= C'_s <= 16, C_s = M C'_s.
 *     Every code must be < K: this is a precondition that the release path
 *     does not report; the kernels clamp a code to K - 1, so a bad code gives
 *     a wrong value but never an access outside the layer's table.  Setting
 *     the environment variable QCNN_CHECK_CODES=1 makes every call verify the
 *     codes first (one extra kernel and a host sync) and return
 *     QCNN_ERR_CODE_RANGE on violation.
 *   - The code array must start at a 4-byte aligned address (any fresh
 *     device allocation does); otherwise QCNN_ERR_UNSUPPORTED.
 *   - Inputs and outputs must not overlap.
 *   - Errors: every argument is validated on the host BEFORE any HIP call;
 *     on a validation error nothing is launched and no output is touched.
 *     Launch or runtime failures return QCNN_ERR_HIP.  No call aborts and no
 *     C++ exception crosses the ABI.
 *   - Execution is asynchronous on `stream` (a hipStream_t; NULL = the legacy
 *     default stream): a call returns once its kernels are enqueued.  Calls
 *     are reentrant.  A conv or FC call that needs temporary device memory
 *     (re-laid-out codes, partial sums) uses a library-owned workspace, one
 *     per (device, stream): grown in stream order on `stream` (the old one
 *     released with hipFreeAsync, a larger one taken from a memory pool the
 *     library creates per device; the device's default pool is not touched),
 *     locked for the enqueue of one call, and held until the process ends.
 *     Concurrent calls on different streams never share it; calls on one
 *     stream use it one after the other in stream order.
 */
#ifndef QCNN_H
#define QCNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum qcnn_status {
  QCNN_OK = 0,
  QCNN_ERR_NULL = 1,        /* a required pointer is NULL */
  QCNN_ERR_SHAPE = 2,       /* a size < 1 (pad < 0), C_s != M C'_s, empty output, overflow */
  QCNN_ERR_K_RANGE = 3,     /* K < 1 or K > 256 */
  QCNN_ERR_CODE_RANGE = 4,  /* a code >= K (only with QCNN_CHECK_CODES=1) */
  QCNN_ERR_HIP = 5,         /* a HIP runtime call or kernel launch failed */
  QCNN_ERR_UNSUPPORTED = 6, /* C'_s > 16, codes not 4-byte aligned, grid or LDS limits */
  QCNN_ERR_ALIAS = 7,       /* an output overlaps an input */
  QCNN_ERR_WORKSPACE = 8    /* qcnn_conv_forward_noalloc: the layer needs more than its static scratch */
} qcnn_status;

/* Build the table of sub-codeword inner products (Sec. 3.1 test phase;
 * Sec. 3.2, table over input positions; Table 1 term d_s^2 C_s K):
 *   lut[n][m][k][y][x] = sum_{j < C'_s} codebooks[m][k][j] * x[n][m C'_s + j][y][x]
 * x: [N][C_s][H][W]; codebooks: [M][K][C'_s]; lut (output): [N][M][K][H][W].
 * A fully-connected input is H = W = 1.  The fused forwards below do not need
 * this table in memory; this entry point exports it. */
qcnn_status qcnn_lut_build(const float* x, int N, int C_s, int H, int W,
                           const float* codebooks, int M, int K, int Csp,
                           float* lut, void* stream);

/* Forward of a PQ convolutional layer, Eq. (7):
 *   y[n][t][yo][xo] = sum_{ky,kx inside} sum_m L[n][m][ codes[t][ky][kx][m] ]
 *                                            [yo stride - pad + ky][xo stride - pad + kx]
 *                     (+ bias[t]) (ReLU)
 * x: [N][C_s][H][W]; codebooks: [M][K][C'_s]; codes: uint8 [C_t][d_k][d_k][M];
 * bias: [C_t] or NULL; y (output): [N][C_t][H_o][W_o].
 * The table is built tile by tile in LDS and never written to memory. */
qcnn_status qcnn_conv_forward(const float* x, int N, int C_s, int H, int W,
                              const float* codebooks, int M, int K, int Csp,
                              const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                              const float* bias, int relu, float* y, void* stream);

/* Forward of a PQ fully-connected layer, Eq. (5):
 *   y[n][t] = sum_m L[n][m][ codes[t][m] ]  (+ bias[t]) (ReLU),
 *   L[n][m][k] = sum_j codebooks[m][k][j] * x[n][m C'_s + j]
 * x: [N][C_s]; codebooks: [M][K][C'_s]; codes: uint8 [C_t][M]; bias: [C_t] or
 * NULL; y (output): [N][C_t]. */
qcnn_status qcnn_fc_forward(const float* x, int N, int C_s,
                            const float* codebooks, int M, int K, int Csp,
                            const uint8_t* codes, int C_t,
                            const float* bias, int relu, float* y, void* stream);

/* qcnn_conv_forward followed by max pooling over pool_k x pool_k windows
 * with stride pool_s and no padding (the pooling between the PQ conv layers
 * of the AlexNet-shaped forward; Sec. 5.2 quantizes such networks layer by
 * layer):
 *   y[n][t][py][px] = max_{dy,dx < pool_k} z[n][t][py pool_s + dy][px pool_s + dx],
 * z the output of qcnn_conv_forward with the same arguments (bias, ReLU),
 * H_p = floor((H_o - pool_k) / pool_s) + 1 (likewise W_p).
 * y (output): [N][C_t][H_p][W_p]; every other argument as in
 * qcnn_conv_forward.  Equal, bit for bit, to qcnn_conv_forward then
 * qcnn_maxpool2d.  A layer whose subspaces are split over workgroups takes
 * the window maxima in the kernel that adds the splits' partial sums, so z
 * never goes to memory; otherwise z lives in the library's workspace.
 * QCNN_ERR_SHAPE for pool_k < 1, pool_s < 1 or an empty pooled map. */
qcnn_status qcnn_conv_pool_forward(const float* x, int N, int C_s, int H, int W,
                                   const float* codebooks, int M, int K, int Csp,
                                   const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                                   const float* bias, int relu, int pool_k, int pool_s,
                                   float* y, void* stream);

/* qcnn_conv_forward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments, limits, kernels and results (bit for bit),
 * but every temporary (re-laid-out codes, partial sums of split layers, the
 * QCNN_CHECK_CODES counter) lives in a static device array of 64 MiB that the
 * library's code object holds on every device it runs on until the process
 * ends; nothing is allocated or freed and no timing events are recorded.  A
 * layer whose temporaries exceed the array returns QCNN_ERR_WORKSPACE before
 * any HIP call (the AlexNet conv3 layer at N = 32 needs about 49 MiB).  The
 * array is shared by every call on a device and keeps the last call's
 * contents: calls that overlap on one device (two streams, or two host
 * threads) race on it, so serialise them. */
qcnn_status qcnn_conv_forward_noalloc(const float* x, int N, int C_s, int H, int W,
                                      const float* codebooks, int M, int K, int Csp,
                                      const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                                      const float* bias, int relu, float* y, void* stream);

/* ---- Prepared layers.  The codes and sub-codebooks of a quantized layer
 * are fixed at test time (Sec. 3.1 and 3.2: the codebooks and quantization
 * indices are stored, and each forward only builds the table and gathers,
 * Eq. (5) / (7)).  A plan takes them once for one input shape: it verifies
 * every code (< K), keeps its own device copies of the codebooks and the
 * bias, and stores the codes in the order the layer's kernel reads them, so
 * that a forward runs only the table build and gather (and, for a layer
 * split over workgroups, the sum of the splits' partial sums);
 * qcnn_conv_forward and qcnn_fc_forward re-lay the codes on every call.
 * Results are those of qcnn_conv_forward (pool_k = pool_s = 0),
 * qcnn_conv_pool_forward (pool_k, pool_s >= 1) or qcnn_fc_forward with the
 * same arguments, bit for bit.  A plan holds no caller pointer: the caller's
 * buffers may be changed or freed once the create call returns.
 *
 * qcnn_conv_plan_create / qcnn_fc_plan_create: arguments as in
 * qcnn_conv_forward / qcnn_fc_forward, without x and y; codes are uint8
 * (packed = 0) or their packed stream (packed = 1, see the packed codes
 * below).  Conv: pool_k = pool_s = 0 for no pooling; pool_k, pool_s >= 1 for
 * max pooling as in qcnn_conv_pool_forward (one of them 0, a negative value
 * or an empty pooled map: QCNN_ERR_SHAPE).  Validation as in the per-call
 * entry points; then one device allocation (hipMalloc) on the current
 * device, the copies and the re-layout on `stream`, a code check
 * (QCNN_ERR_CODE_RANGE if a code is >= K, whatever QCNN_CHECK_CODES says),
 * and a synchronisation of `stream`.  On success *plan is the new plan; on
 * any error nothing is left allocated and *plan is not written.  The conv
 * kernel is chosen at creation (QCNN_CONV_KERNEL as read then).
 *
 * qcnn_plan_forward: x of the plan's input shape ([N][C_s][H][W], FC
 * [N][C_s]); y (output) [N][C_t][H_o][W_o], pooled [N][C_t][H_p][W_p], FC
 * [N][C_t]; on the device the plan was created on (else
 * QCNN_ERR_UNSUPPORTED); x and y must not overlap (QCNN_ERR_ALIAS).
 * Asynchronous on `stream`; temporaries (partial sums, a full map to pool)
 * come from the library's per-stream workspace as for the per-call entry
 * points.  Forwards of one plan on several streams may run concurrently
 * (the plan is only read).
 *
 * qcnn_plan_destroy: waits for the plan's device to finish its work, then
 * frees the plan; NULL is accepted. */
typedef struct qcnn_plan qcnn_plan;

qcnn_status qcnn_conv_plan_create(int N, int C_s, int H, int W,
                                  const float* codebooks, int M, int K, int Csp,
                                  const uint8_t* codes, int packed, int C_t, int d_k, int stride, int pad,
                                  const float* bias, int relu, int pool_k, int pool_s,
                                  qcnn_plan** plan, void* stream);
qcnn_status qcnn_fc_plan_create(int N, int C_s,
                                const float* codebooks, int M, int K, int Csp,
                                const uint8_t* codes, int packed, int C_t,
                                const float* bias, int relu, qcnn_plan** plan, void* stream);
qcnn_status qcnn_plan_forward(const qcnn_plan* plan, const float* x, float* y, void* stream);
qcnn_status qcnn_plan_destroy(qcnn_plan* plan);

/* ---- Packed codes.  Table 1 (Sec. 3.4) stores every quantization index in
 * log2 K bits: (1/8) d_k^2 M C_t log2 K bytes for a conv layer,
 * (1/8) M C_t log2 K for a fully-connected one.  The packed form is a bit
 * stream of b = qcnn_code_bits(K) bits per code (b = 0 for K = 1, else the
 * smallest b with 2^b >= K, i.e. log2 K for a power of two): code i of the
 * array, in the array's own order ([C_t][d_k][d_k][M] or [C_t][M]), is
 * stream bits i b .. i b + b - 1 with value bit j at stream bit i b + j, and
 * stream bit q is bit q % 8 of byte q / 8 (least significant bit first).
 * A packed buffer is qcnn_packed_bytes(n, K) = 4 ceil(n b / 32) bytes: the
 * ceil(n b / 8) bytes of the stream, then zero bits up to a whole dword.
 * Buffers are device pointers, 4-byte aligned (else QCNN_ERR_UNSUPPORTED).
 * The codes must be < K (the precondition of the forward); packing keeps the
 * low b bits of each code.  With QCNN_CHECK_CODES=1 qcnn_pack_codes verifies
 * its input first. */

/* Bits per packed code for K sub-codewords, or -1 when K is outside [1, 256]. */
int qcnn_code_bits(int K);

/* Size in bytes of the packed form of n codes (0 when K is outside [1, 256]). */
size_t qcnn_packed_bytes(size_t n, int K);

/* codes: uint8 [n] -> packed (output): qcnn_packed_bytes(n, K) bytes. */
qcnn_status qcnn_pack_codes(const uint8_t* codes, size_t n, int K, uint8_t* packed, void* stream);

/* packed: qcnn_packed_bytes(n, K) bytes -> codes (output): uint8 [n]. */
qcnn_status qcnn_unpack_codes(const uint8_t* packed, size_t n, int K, uint8_t* codes, void* stream);

/* qcnn_conv_forward and qcnn_fc_forward with the codes in packed form
 * (qcnn_packed_bytes of C_t d_k^2 M or C_t M codes).  Same arguments, limits
 * and results: for the same codes the outputs are identical bit for bit. */
qcnn_status qcnn_conv_forward_packed(const float* x, int N, int C_s, int H, int W,
                                     const float* codebooks, int M, int K, int Csp,
                                     const uint8_t* packed_codes, int C_t, int d_k, int stride, int pad,
                                     const float* bias, int relu, float* y, void* stream);
qcnn_status qcnn_fc_forward_packed(const float* x, int N, int C_s,
                                   const float* codebooks, int M, int K, int Csp,
                                   const uint8_t* packed_codes, int C_t,
                                   const float* bias, int relu, float* y, void* stream);

/* ---- Parameter quantization (the step that produces codebooks and codes).
 * Sec. 3.1, Eq. (4): for each subspace m, minimise || D^(m) B^(m) - W^(m) ||_F^2
 * over the K sub-codewords D^(m) and the indicator columns B^(m), by k-means
 * over the sub-vectors; Sec. 3.2, Eq. (6): a conv layer shares D^(m) over all
 * kernel positions p_k, so subspace m's k-means runs over the sub-vectors of
 * every (c_t, p_k).
 * W: [C_t][C_s][d_k][d_k] fp32 (a fully-connected layer is d_k = 1, W[c_t][c_s]);
 * the sub-vector of (c_t, p_k, m) is W[c_t][m C'_s + j][p_k], j < C'_s.
 * codebooks: [M][K][C'_s]; codes: uint8 [C_t][d_k][d_k][M] (FC: [C_t][M]),
 * the layouts qcnn_conv_forward / qcnn_fc_forward read.
 * Assignment: the nearest sub-codeword in squared Euclidean distance,
 * accumulated in fp32 as d = fma(w_j - c_j, w_j - c_j, d) over j in order,
 * the first minimum winning (ties go to the lowest index).  Update: each
 * sub-codeword becomes the mean of its sub-vectors, summed in float64 in
 * sub-vector order (c_t, p_k) and rounded to fp32; one that no sub-vector
 * chose keeps its value.  Objectives are float64 sums of the fp32 minimum
 * distances.  Limits as for the forward: 1 <= K <= 256, C'_s <= 16, C_s =
 * M C'_s, M <= 65535.  All pointers are device pointers; inputs and outputs
 * must not overlap (codebooks are updated in place where stated). */

/* One assignment.  codes (output); objective (output, nullable): [M] float64,
 * per subspace the sum of the minimum distances. */
qcnn_status qcnn_pq_assign(const float* W, int C_t, int C_s, int d_k,
                           const float* codebooks, int M, int K, int Csp,
                           uint8_t* codes, double* objective, void* stream);

/* One update from given codes (every code must be < K): codebooks is read
 * and replaced in place; counts (output, nullable): int [M][K], sub-vectors
 * per sub-codeword. */
qcnn_status qcnn_pq_update(const float* W, int C_t, int C_s, int d_k,
                           const uint8_t* codes, int M, int K, int Csp,
                           float* codebooks, int* counts, void* stream);

/* k-means: iters x (assignment, update), then a final assignment, so that
 * the codes match the returned sub-codewords.  codebooks: in, the initial
 * sub-codewords (the caller draws them); out, the learned ones.  codes
 * (output); objective (output, nullable): [iters + 1] float64, the total
 * over m after each assignment.  iters >= 0. */
qcnn_status qcnn_pq_kmeans(const float* W, int C_t, int C_s, int d_k,
                           int M, int K, int Csp, int iters,
                           float* codebooks, uint8_t* codes, double* objective, void* stream);

/* ---- Error-corrected quantization of a fully-connected layer (Sec. 3.3.1).
 * Minimises the response error of Eq. (8),
 *   sum_n || T_n - sum_m (D^(m) B^(m))^T S_n^(m) ||^2,
 * over the sub-codebooks and assignments by block coordinate descent over
 * the subspaces: for subspace m, with R^(m) the residual of the others
 * (Eq. (9)), `inner` rounds of the sub-codebook update of Eq. (11) (each
 * sub-codeword the least-squares fit over the images and the output
 * channels assigned to it) then the assignment update of Eq. (12) (each
 * channel the sub-codeword of least residual error).  A call runs `sweeps`
 * sweeps over m = 0 .. M-1 in order, starting from the codebooks and codes
 * given (normally those of qcnn_pq_kmeans).
 * S: [N][C_s] the layer's inputs; T: [N][C_t] the desired responses (fp32);
 * codebooks [M][K][C'_s] fp32 and codes uint8 [C_t][M]: updated in place;
 * objective (output, nullable): [1 + sweeps M] float64, Eq. (8) before the
 * first step and after every subspace step (non-increasing up to rounding).
 * Arithmetic is float64 throughout (the residual E = T - S W-hat is kept in
 * a library workspace of 8 N C_t bytes plus partial sums); the codebooks
 * are rounded to fp32 once at the end.  A sub-codeword no channel uses keeps
 * its value; the normal equations |L_k| G D_k = sum_{c in L_k} S^(m)T r_c,
 * G = S^(m)T S^(m), are solved by elimination in channel order, a pivot
 * <= 1e-12 x max diag(G) (a direction the inputs do not span, such as a
 * channel that is zero on every image) setting that coordinate to 0;
 * assignment ties go to the lowest index.  Limits: those of the forward,
 * N <= 2^20, C_t <= 65536; codes >= K are read, and written back, as K - 1
 * (checked with QCNN_CHECK_CODES=1). */
qcnn_status qcnn_ec_fc(const float* S, int N, int C_s, const float* T, int C_t,
                       float* codebooks, int M, int K, int Csp, uint8_t* codes,
                       int sweeps, int inner, double* objective, void* stream);

/* ---- Error-corrected quantization of a convolutional layer (Sec. 3.3.2
 * Eq. (13); App. B Eq. (14)-(21)).  Minimises the response error
 *   sum_{n, p_t} || sum_{(p_k, p_s)} sum_m (D^(m) B^(m)_{p_k})^T S^(m)_{n, p_s} - T_{n, p_t} ||^2
 * by block coordinate descent over the subspaces; for subspace m, with the
 * residual of the others (Eq. (15)), `inner` rounds of: the sub-codewords
 * k = 0 .. K-1 in order, each the least-squares fit of Eq. (19) to the
 * residual without the other sub-codewords' terms (Eq. (18)); then the
 * kernel positions in row-major order, each channel taking the sub-codeword
 * of least error for the residual without the other positions' terms
 * (Eq. (20)-(21)).  Each step uses the latest values of the others.
 * Readings of the appendix's garbled indices: Eq. (18) takes out, per
 * channel, the positions whose sub-codeword is not k, and Eq. (19) sums over
 * the channels that have a position on k; Eq. (20) takes out every other
 * position p'_k with its own input position p'_s.  p_s = p_t stride - pad +
 * p_k (no flip), S = 0 outside the input.
 * S: [N][C_s][H][W] inputs; T: [N][C_t][H_o][W_o] desired responses (fp32);
 * codebooks [M][K][C'_s] fp32 and codes uint8 [C_t][d_k][d_k][M] (the
 * forward's layouts): updated in place; objective (output, nullable):
 * [1 + sweeps M] float64, the error before the first step and after every
 * subspace step.  Arithmetic is float64 (a workspace of 8 N C_t H_o W_o
 * bytes plus small per-subspace arrays); normal equations solved as in
 * qcnn_ec_fc (elimination in channel order, a pivot <= 1e-12 x the largest
 * diagonal entry dropping that coordinate); a sub-codeword that no position
 * uses keeps its value; ties go to the lowest index.  Limits: C'_s <= 8,
 * C_t d_k^2 <= 16384, N C_t H_o W_o <= 2^31; codes >= K are read, and
 * written back, as K - 1 (checked with QCNN_CHECK_CODES=1).  Cost per call:
 * M d_k^4 C'_s^2 N H_o W_o multiply-adds once for the input Gram blocks,
 * then per subspace step two passes over the residual and a one-workgroup
 * solve that is sequential over the K sub-codewords. */
qcnn_status qcnn_ec_conv(const float* S, int N, int C_s, int H, int W,
                         const float* T, int C_t, int d_k, int stride, int pad,
                         float* codebooks, int M, int K, int Csp, uint8_t* codes,
                         int sweeps, int inner, double* objective, void* stream);

/* Network glue between PQ layers (not part of the paper's method): max
 * pooling over k x k windows with stride s and no padding,
 *   y[n][c][yo][xo] = max_{dy,dx < k} x[n][c][yo s + dy][xo s + dx],
 * H_o = floor((H - k) / s) + 1.  x: [N][C][H][W]; y (output): [N][C][H_o][W_o]. */
qcnn_status qcnn_maxpool2d(const float* x, int N, int C, int H, int W, int k, int s,
                           float* y, void* stream);

/* Output size of a conv / pool along one axis (0 if empty).  Host only. */
int qcnn_out_size(int in, int k, int stride, int pad);

/* Static description of a status code.  Host only; never NULL. */
const char* qcnn_status_string(qcnn_status s);

/* ABI version, currently 1. */
int qcnn_version(void);

/* Kernel timing, for benchmarks and profiling.  While enabled, every
 * compute call above times its main kernel (the gather kernel of
 * qcnn_conv_forward and qcnn_fc_forward, the table kernel of
 * qcnn_lut_build) with a pair of HIP events that the kernel's dispatch
 * stamps at the start and the end of its execution (hipExtLaunchKernelGGL),
 * so the pair measures the kernel alone; the quantizer calls record a pair
 * on their stream around their kernels (the assignment or update kernels of
 * qcnn_pq_assign / qcnn_pq_update, the whole iteration loop of
 * qcnn_pq_kmeans).  Code re-layout and split-sum kernels are outside the
 * pairs.  Off by default; when off the calls create no events.  Enabling
 * and disabling are process-wide and take effect for later calls. */
qcnn_status qcnn_timing_enable(int enable);

/* Waits for every pair recorded since the last read, returns their summed
 * elapsed milliseconds in *total_ms and their number in *launches, then
 * destroys them.  QCNN_ERR_NULL if an argument is NULL; QCNN_ERR_HIP if an
 * event could not be created, recorded or read (the sums then cover the
 * readable pairs only). */
qcnn_status qcnn_timing_read(double* total_ms, long long* launches);

/* The same drain with each pair's elapsed milliseconds, in launch order,
 * written to ms_each[0 .. min(*launches, capacity)); *launches is the number
 * of pairs read (all are destroyed, also those past `capacity`). */
qcnn_status qcnn_timing_read_each(double* ms_each, long long capacity, long long* launches);

/* Peak probes, for the benchmark's roofline denominators (not part of the
 * paper's method).  Both synchronise with `stream` and allocate small
 * temporaries.
 * qcnn_probe_lds: every CU of the current device streams conflict-free
 * 128-bit LDS reads (one 1024-thread workgroup per CU, each wave reading
 * 1 KB contiguous runs); returns the LDS read bytes per clock per CU, the
 * shader clock in GHz measured under that load (shader-clock counter over
 * the constant-rate counter), and the aggregate bytes per second.
 * qcnn_probe_hbm: streams `bytes` (a multiple of 16 is used) of the device
 * buffer src with 16-byte loads, then fills dst with 16-byte stores, then
 * copies src to dst; returns the read rate, the write rate and the copy rate
 * (bytes read + written per second).  src and dst: 16-byte aligned, `bytes`
 * long each, not overlapping; dst is overwritten. */
qcnn_status qcnn_probe_lds(double* bytes_per_clk_cu, double* clock_ghz, double* bytes_per_s, void* stream);
qcnn_status qcnn_probe_hbm(const void* src, void* dst, size_t bytes, double* read_bytes_per_s,
                           double* write_bytes_per_s, double* copy_bytes_per_s, void* stream);

/* VALU issue probe: 16 waves per CU on every CU, each issuing independent
 * streams of one instruction kind; returns the shader clocks per wave64
 * instruction per SIMD of v_add_f32, of v_add_f32 with a DPP wave_shl:1
 * operand, and of v_mad_u32_u24 (the instructions a table read of the conv
 * gather issues). */
qcnn_status qcnn_probe_valu(double* add_clk, double* dpp_add_clk, double* mad_clk, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QCNN_H */
