/*
 * qmlp.h -- C ABI of the MI355X (gfx950) W4/W2-GateUp decode-MLP library.
 *
 * The library runs the inference hot path of the W4/W2-GateUp deployment
 * with Recover-LoRA adapters (arXiv 2606.04238): one gated-MLP block whose
 * gate and up projections are 2-bit group-quantized, each carrying an
 * unmerged low-rank correction x A^T B^T, followed by SiLU(gate) * up and a
 * 4-bit group-quantized down projection.
 *
 *   Sec. 3.1, Eq. (1)  LoRA-augmented linear  Y = W X + alpha B A X.
 *   Sec. 3.3           W4/W2-GateUp: gate/up at 2 bits, every other linear
 *                      (down included) at 4 bits, group-wise quantization.
 *   Sec. 4.1           Stage 1: gate/up to INT2 by post-training quantization.
 *   Sec. 4.2           adapters on the quantized gate/up, kept as a separate
 *                      module at inference (not merged into the 2-bit grid).
 *   Sec. 5             the MLP is one fused gate-activation-down operator;
 *                      decode is bound by the bandwidth of loading weights.
 *   Sec. 7             deployment: quantize gate/up to INT2 (step 1), the rest
 *                      to INT4 (step 4), deploy with attached adapters (step 5).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer except the qmlp_qweight/qmlp_mlp descriptors and the
 *    status-string result is a DEVICE pointer into memory the caller owns.
 *    The library never allocates or frees device memory and keeps no pointer
 *    after a call returns.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *    and runs asynchronously; nothing synchronizes.
 *  - Arguments are validated first.  On any error nothing is enqueued and no
 *    output is written.  A HIP launch error maps to QMLP_ERR_HIP; a fault
 *    inside a kernel surfaces at the caller's next synchronization.
 *  - Calls are reentrant: there is no global mutable state.  Inputs and
 *    outputs of one call must not overlap.
 *
 * Storage format of a quantized matrix W [n][k] (nn.Linear orientation:
 * n outputs, k inputs; groups of g consecutive inputs of one row):
 *  - codes: row-major, each row a run of little-endian 32-bit words; code i
 *    of a row sits at bits [b*(i mod 32/b), +b) of word i/(32/b) of that row
 *    (16 codes per word at b=2, 8 at b=4).  Size n*k*b/8 bytes.
 *    At b=3 (Appendix B) a row is two planes: the low two bits of every code
 *    in the 2-bit layout (k/16 words), then the high bit of every code, code
 *    i at bit (i mod 32) of word i/32 of that plane (k/32 words); k % 128 == 0
 *    (rows of 3k/8 bytes stay 16-byte aligned).
 *  - meta: row-major [n][k/g] pairs of binary16 (scale, zero), scale first.
 *    Size n*(k/g)*4 bytes.  The dequantized weight is scale * (q - zero).
 *  - Quantizer (round-to-nearest, asymmetric min-max; the paper fixes only
 *    the bit width and grouping): per group lo = min(0, min w),
 *    hi = max(0, max w), s = (hi - lo)/(2^b - 1) in fp64, scale = s rounded
 *    once to binary16 (nearest-even; 0 becomes 1.0),
 *    zero = clamp(rint(-lo/scale), 0, 2^b - 1) (an integer),
 *    q = clamp(rint(w/scale) + zero, 0, 2^b - 1); rint is nearest-even and
 *    every quotient an IEEE fp64 division.
 *
 * Activation types: x, h, y and the LoRA factors are binary16 (QMLP_F16) on
 * the decode path (1 <= M <= 16) and bfloat16 (QMLP_BF16) on the
 * prefill-chunk path (M a multiple of 128); accumulation is fp32.
 */
#ifndef QMLP_H
#define QMLP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    QMLP_OK = 0,
    QMLP_ERR_NULL = 1,          /* a required pointer is NULL */
    QMLP_ERR_SHAPE = 2,         /* sizes inconsistent or not a supported multiple */
    QMLP_ERR_ALIGN = 3,         /* a device pointer is not 16-byte aligned */
    QMLP_ERR_UNSUPPORTED = 4,   /* bits / group / rank / M / dtype combination not built */
    QMLP_ERR_WORKSPACE = 5,     /* workspace NULL or smaller than qmlp_workspace_bytes() */
    QMLP_ERR_HIP = 6            /* a HIP runtime call failed (launch, attribute, device query) */
} qmlp_status;

typedef enum { QMLP_F16 = 0, QMLP_BF16 = 1 } qmlp_dtype;

/* A hipStream_t passed as an opaque pointer (NULL = the null stream). */
typedef void *qmlp_stream;

/* Non-owning view of one packed quantized matrix in device memory. */
typedef struct {
    int32_t bits;     /* 2 (gate/up) or 4 (down); 3 for gate/up; see qmlp_mlp */
    int32_t n_out;    /* rows n of the logical W [n][k] */
    int32_t k_in;     /* columns k; groups run along k */
    int32_t group;    /* g: 32, 64 or 128; k_in % g == 0 */
    void *codes;      /* qmlp_codes_bytes(bits, n_out, k_in) bytes, 16-B aligned */
    void *meta;       /* qmlp_meta_bytes(n_out, k_in, group) bytes, 16-B aligned */
} qmlp_qweight;

/* One W4/W2-GateUp MLP block with its Recover-LoRA adapters (Sec. 3.3, 4.2).
 * gate/up at 2 bits and down at 4 bits, groups of 64 or 128, is the block
 * every path takes.  The binary16 decode path (qmlp_forward,
 * qmlp_forward_layers, qmlp_forward_batch; not the one-kernel layer, the
 * streamed and matrix-core launches nor the persistent stack, which take
 * only that form) also runs the comparison
 * points of the throughput analysis (Sec. 5.2) and the paper's INT2 grouping
 * (Sec. 3.3, Sec. 4.1): gate/up at 4 bits (uniform W4), down at 2 bits
 * (uniform W2, groups of 64 or 128), and group 32 for gate/up (any width)
 * and for a 4-bit down; and the 3-bit gate/up of Appendix B (W3, group 32
 * in the paper; 64 and 128 also accepted). */
typedef struct {
    qmlp_qweight gate;      /* bits 2 (or 3, 4), [f][d] */
    qmlp_qweight up;        /* same bits and group as gate, [f][d] */
    qmlp_qweight down;      /* bits 4 (or 2), [d][f] */
    const void *A_gate;     /* [rank][d] activation type (nn.Linear / PEFT "lora_A") */
    const void *B_gate;     /* [f][rank] activation type (PEFT "lora_B")            */
    const void *A_up;       /* [rank][d] */
    const void *B_up;       /* [f][rank] */
    int32_t rank;           /* r: 0 (no adapter), 8, 16 or 32 */
    float lora_scale;       /* multiplies B A x (Eq. (1)'s alpha; PEFT: alpha/r) */
} qmlp_mlp;

/* ---------------------------------------------------------------- sizes */

/* Bytes of packed codes for an [n_out][k_in] matrix at `bits` (0 if invalid). */
size_t qmlp_codes_bytes(int bits, int n_out, int k_in);

/* Bytes of (scale, zero) metadata for [n_out][k_in] at group `group` (0 if invalid). */
size_t qmlp_meta_bytes(int n_out, int k_in, int group);

/* Workspace bytes qmlp_forward / qmlp_gateup_w2_lora need for this block at
 * M tokens (0 if the combination is unsupported).  Layout: a 1024-byte
 * control block (uint32 words, each on its own 128-byte line: word 0 counts
 * the one-kernel layer's calls, word 32 its finished blocks, word 160 holds
 * sticky error bits: 1 = t wait timed out, 2 = h wait timed out), then t
 * (fp32), h (activation type [M][f]), on the prefill path lora_scale * t in
 * bfloat16, and on the decode path the one-kernel layer's tagged hand-off
 * words (one [4][64] block of 64-bit words per compute unit, [4][f] 32-bit),
 * and on the prefill path, when the down projection splits f into slices
 * to fill the chip, the slices' fp32 partial sums [S][M][d].  The workspace must be ZERO before
 * its first call, and zeroed again before it serves a block of another shape
 * or after an error bit appeared (the results of that call are invalid).
 * One workspace serves one call at a time: calls that overlap in time on the
 * same workspace race. */
size_t qmlp_workspace_bytes(const qmlp_mlp *mlp, int M, qmlp_dtype dtype);

/* ----------------------------------------------------- packing (offline) */

/*
 * Sec. 4.1 / Sec. 7 step 1: quantize fp32 W [n_out][k_in] (row-major,
 * device) to 2-bit codes, group `group` along k_in, writing out->codes and
 * out->meta (caller-allocated, sizes from qmlp_codes_bytes/qmlp_meta_bytes).
 * On success out->bits/n_out/k_in/group are filled in.
 * A group holding a non-finite weight or whose scale overflows binary16 is
 * written as codes 0, scale NaN (0x7E00), zero 0, and bit 0 of *d_status
 * (a device int32, may be NULL) is set with an atomic OR; the caller zeroes
 * *d_status beforehand.  Requires group in {32, 64, 128}, k_in % group == 0
 * (32 is the paper's INT2 group).
 */
qmlp_status qmlp_pack_w2(const float *W, int n_out, int k_in, int group,
                         qmlp_qweight *out, int32_t *d_status, qmlp_stream stream);

/* Appendix B: the same at 3 bits (the W3 gate/up variant), in the two-plane
 * layout above.  Requires group in {32, 64, 128}, k_in % 128 == 0. */
qmlp_status qmlp_pack_w3(const float *W, int n_out, int k_in, int group,
                         qmlp_qweight *out, int32_t *d_status, qmlp_stream stream);

/* Sec. 3.3 / Sec. 7 step 4: the same at 4 bits (down projection and every
 * other non-gate/up linear).  Requires group in {32, 64, 128}, k_in % group == 0. */
qmlp_status qmlp_pack_w4(const float *W, int n_out, int k_in, int group,
                         qmlp_qweight *out, int32_t *d_status, qmlp_stream stream);

/* ------------------------------------------------------ the hot path */

/*
 * Sec. 3.1 Eq. (1) on the gate and up projections, then the activation of
 * the fused gate-activation-down operator (Sec. 5):
 *   G = W2gate x + lora_scale * B_gate (A_gate x)
 *   U = W2up   x + lora_scale * B_up   (A_up   x)
 *   h = SiLU(G) * U = G / (1 + exp(-G)) * U
 * x [M][d] and h [M][f] are row-major in the activation type `dtype`.
 * ws/ws_bytes: workspace of at least qmlp_workspace_bytes(mlp, M, dtype).
 * M == 0 enqueues nothing and returns QMLP_OK.  Gate and up must be 2-bit
 * (group 32 allowed on the decode path); QMLP_ERR_UNSUPPORTED otherwise.
 */
qmlp_status qmlp_gateup_w2_lora(const qmlp_mlp *mlp, const void *x, int M, qmlp_dtype dtype,
                                void *h, void *ws, size_t ws_bytes, qmlp_stream stream);

/*
 * The 4-bit down projection (Sec. 3.3): y [M][n_out] = W4down h, with
 * h [M][k_in] and y row-major in the activation type.  No workspace.
 * Group 32 only on the binary16 decode path.
 */
qmlp_status qmlp_down_w4(const qmlp_qweight *down, const void *h, int M, qmlp_dtype dtype,
                         void *y, qmlp_stream stream);

/*
 * The whole block, y = W4down(SiLU(G) * U) (Sec. 3.3, 4.2, 5), x [M][d] ->
 * y [M][d].  The intermediate h lives only in the workspace.
 */
qmlp_status qmlp_forward(const qmlp_mlp *mlp, const void *x, int M, qmlp_dtype dtype,
                         void *y, void *ws, size_t ws_bytes, qmlp_stream stream);

/*
 * qmlp_forward without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The block's workspace is a fixed array
 * of qmlp_noalloc_scratch_bytes() (1 MiB) in this library's device memory,
 * one per GPU, held until the process ends; the call allocates and frees
 * nothing.  Binary16 decode only (1 <= M <= 16): QMLP_ERR_UNSUPPORTED for
 * bfloat16, QMLP_ERR_WORKSPACE when qmlp_workspace_bytes(mlp, M, dtype)
 * exceeds the array (the Qwen3-4B, Qwen3-8B and 14B-class blocks fit up to
 * M = 16; d = 8192, f = 32768 fits up to M = 7).  Each call first clears the part of the array
 * the block uses (one small fill kernel, then the kernels of qmlp_forward,
 * on `stream`), so it never depends on an earlier call's contents.  All
 * calls on one GPU share its array: calls that overlap in time on the same
 * GPU (other streams, other host threads) race.  Other errors as for
 * qmlp_forward; on any error nothing is enqueued.
 */
qmlp_status qmlp_forward_noalloc(const qmlp_mlp *mlp, const void *x, int M, qmlp_dtype dtype,
                                 void *y, qmlp_stream stream);

/* Size of the per-GPU array behind qmlp_forward_noalloc.  Host-only. */
size_t qmlp_noalloc_scratch_bytes(void);

/*
 * A stack of L blocks of one shape on a residual stream, as the MLP
 * sub-blocks of an L-layer decoder with the attention sub-blocks left out
 * (Sec. 3.3: each layer carries one gated MLP):
 *   x_0 = x,  u_l = RMSNorm(x_l),  y_l = block_l(u_l),  x_{l+1} = x_l + y_l,
 * RMSNorm(v) = v / sqrt(mean(v^2) + 1e-6) per token with unit gain (a
 * learned gain folds into the input columns of gate, up and LoRA-A before
 * quantization).  u_l and y_l are rounded to binary16, the sum of two
 * binary16 values is rounded once (nearest-even).  Binary16 only.
 * layers[0..L-1] are host descriptors (same d, f, group and rank); x [M][d];
 * y [L][M][d] receives every block's output (layer l at y + l*M*d); x_out
 * [M][d] (may be NULL) receives x_L.  Each y_l equals qmlp_forward of layer
 * l on RMSNorm(x_l) within the output bar.
 *
 * At M = 1 for shapes with f % 256 == 0, d % 512 == 0, d <= 4096,
 * (d/g) % 4 == 0 on a GPU with 8 XCDs of 32 compute units, the stack runs
 * as ONE persistent launch per 40 layers: the weights of block l+1 stream in
 * while block l finishes (weights do not depend on activations), and no
 * step of block l+1 starts before x_{l+1} is complete.  Every other shape
 * runs per block: a norm kernel, qmlp_forward, a residual-add kernel.
 *
 * ws/ws_bytes: at least qmlp_stack_workspace_bytes(layers, L, M, dtype),
 * zero before the first call, with the rules of qmlp_workspace_bytes (after
 * the per-block workspace come three activation buffers, then the
 * persistent launch's 1024-byte control block -- word 0 its step counter,
 * word 64 sticky error bits: 1/2/4 = a wait for the activation / h / the
 * cross-XCD partials gave up, 8 = a workgroup found no place -- and its
 * hand-off words).  Errors as for qmlp_forward; QMLP_ERR_UNSUPPORTED for
 * bfloat16.
 */
size_t qmlp_stack_workspace_bytes(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

qmlp_status qmlp_forward_stack(const qmlp_mlp *layers, int L, const void *x, int M,
                               qmlp_dtype dtype, void *y, void *x_out, void *ws, size_t ws_bytes,
                               qmlp_stream stream);

/* Byte offset, within a qmlp_forward_stack workspace, of the persistent
 * launch's sticky error word (a uint32: 1/2/4 = a wait for the activation /
 * h / the cross-XCD partials gave up, 8 = a workgroup had no place; the
 * word is cleared by the caller when it zeroes the workspace and never by
 * the library); 0 if these blocks do not run persistently or the call would
 * be rejected.  Host-only. */
size_t qmlp_stack_error_offset(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

/* Launches qmlp_forward_stack makes: the number of persistent launches when
 * the stack runs persistently, else the per-layer kernels plus the norm and
 * residual-add kernels; 0 if the call would be rejected.  Host-only. */
int qmlp_stack_launches(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

/*
 * L independent blocks of one shape (Sec. 3.3, 4.2, 5: the gated MLP of each
 * layer of the modelled decoders, with separately seeded weights and
 * inputs): y_l = block_l(x_l) for l = 0..L-1, each exactly the operation of
 * qmlp_forward.  layers[0..L-1] are host descriptors (same d, f, group and
 * rank); x [L][M][d] and y [L][M][d] are row-major in the activation type
 * (block l at x + l*M*d, y + l*M*d).
 *
 * Binary16 blocks run in batches of up to 40.  At M = 1 in the
 * W4/W2-GateUp form (2-bit gate/up, 4-bit down, groups 64/128, rank 0, 8,
 * 16 or 32) with d % 512 == 0, d <= 4096, f % 128 == 0, f <= 12288, a batch
 * STREAMS: the LoRA-A products of every block (one launch), then one
 * persistent gate/up launch and one persistent down launch, each workgroup
 * owning a contiguous range of the batch's rows flattened over blocks, so
 * no workgroup waits for another and h of every block passes through the
 * workspace between the two launches.  At 3 <= M <= 16 in the same form
 * (d % 512 == 0, f % 256 == 0, and the LDS limits qmlp_layers_path
 * reports) a batch runs on the MATRIX CORES: the LoRA-A launch (fp32
 * partial sums over four slices of d, added in slice order by the next
 * launch), then one persistent gate/up launch and one persistent down
 * launch that multiply every unpacked weight into all M tokens with
 * v_mfma_f32_16x16x32_f16.  Every other binary16 batch runs the
 * stand-alone kernels as qmlp_forward_batch does; bfloat16 runs
 * qmlp_forward once per block.
 *
 * ws/ws_bytes: at least qmlp_layers_workspace_bytes(layers, L, M, dtype)
 * (binary16: that of qmlp_forward_batch, with four times its t area on the
 * matrix cores and twice on the streamed path).  On the streamed path with
 * adapters the gate/up launch also computes LoRA-A and hands t over as
 * tagged words: the control block's word 0 counts the calls and word 160
 * holds sticky error bits (1 = a wait for t gave up), so the workspace must
 * be ZERO before its first call and zeroed again before it serves other
 * blocks' shape or after an error bit; one call at a time per workspace.
 * The other paths keep no state between calls.
 * Errors as for qmlp_forward.
 */
size_t qmlp_layers_workspace_bytes(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

qmlp_status qmlp_forward_layers(const qmlp_mlp *layers, int L, const void *x, int M,
                                qmlp_dtype dtype, void *y, void *ws, size_t ws_bytes,
                                qmlp_stream stream);

/* Which path qmlp_forward_layers takes for these blocks: 1 = streamed, 2 =
 * the batched stand-alone kernels, 3 = qmlp_forward per block (bfloat16),
 * 4 = matrix cores; 0 if the call would be rejected.  Host-only (it queries
 * the current device's compute-unit count). */
int qmlp_layers_path(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

/* Launches qmlp_forward_layers makes: per batch of up to 40 blocks 2 on the
 * streamed path, 3 on the matrix-core and batched paths (2 without
 * adapters), or the per-block launches of qmlp_forward; 0 if the call would
 * be rejected.  Host-only. */
int qmlp_layers_launches(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

/*
 * The same L independent blocks as qmlp_forward_layers, always on the
 * stand-alone decode kernels, in batches of up to 40 blocks: the LoRA-A
 * products of every block of a batch (one launch, skipped at rank 0), then
 * gate/up with SiLU(G) * U of every block (one launch), then down of every
 * block (one launch).  Binary16 only (1 <= M <= 16), any width combination
 * qmlp_mlp lists: it is the path of the width comparison (Sec. 5.2), where
 * every precision must run on the same kernels, and of callers that do not
 * want a launch holding every compute unit.  h and t of a batch stay in the
 * workspace between the launches.
 *
 * ws/ws_bytes: at least qmlp_batch_workspace_bytes(layers, L, M, dtype):
 * a 1024-byte block left at zero, t [min(L,40)][M][2r] fp32, h
 * [min(L,40)][M][f] binary16.  No state is kept between calls.  Errors as
 * for qmlp_forward_layers; QMLP_ERR_UNSUPPORTED for bfloat16.
 */
size_t qmlp_batch_workspace_bytes(const qmlp_mlp *layers, int L, int M, qmlp_dtype dtype);

qmlp_status qmlp_forward_batch(const qmlp_mlp *layers, int L, const void *x, int M,
                               qmlp_dtype dtype, void *y, void *ws, size_t ws_bytes,
                               qmlp_stream stream);

/*
 * L independent group-quantized linears of one shape, y_l = W_l x_l (Sec. 3.3:
 * every linear outside gate/up is INT4 in W4/W2-GateUp; at 2 bits they are
 * the uniform-W2 comparison point of Sec. 5.2): the attention projections of
 * a decoder layer (q, k and v as one [q+2kv][d] matrix, o) and the LM head.
 * w[0..L-1] are host descriptors of one shape [n][k] and width (4, or 2 with
 * group 64/128), 1 <= L <= 40; x [L][M][k] and y [L][M][n] binary16,
 * 1 <= M <= 16 (M == 0 is a no-op).  One launch of the stand-alone down
 * kernel over the batch; no workspace.  n % 64 == 0, k % 64 == 0.
 */
qmlp_status qmlp_linear_batch(const qmlp_qweight *w, int L, const void *x, int M,
                              qmlp_dtype dtype, void *y, qmlp_stream stream);

/*
 * The MLP of a mixture-of-experts decoder layer at decode (Sec. 5: the
 * routed experts of the GPT-OSS-20B-class model; only the routed experts'
 * weights are read per token): each of E experts is one block of
 * qmlp_forward (W4/W2-GateUp with its own adapters, or any width qmlp_mlp
 * lists), and token m's output is
 *     y[m] = sum_j topk_w[m][j] * expert_{topk_idx[m][j]}(x[m]).
 * experts[0..E-1]: host descriptors of one shape, 1 <= E <= 40.  x [M][d],
 * y [M][d] binary16; topk_idx int32 [M][k] and topk_w fp32 [M][k] are DEVICE
 * arrays (routing runs on the GPU); ids outside [0, E) are a precondition
 * violation (the kernels clamp them, so nothing is read outside the
 * table).  1 <= k <= E, M <= 16, M*k <= 40.  Every (token, slot) pair runs
 * as one instance: an expert chosen by two tokens is read twice.  Two
 * launches over the M*k instances: gate/up, whose first workgroups of each
 * instance compute LoRA-A (with adapters) and hand t to the others as tagged
 * words, then down.  With
 * k <= 4 (and h of the k instances within the down kernel's LDS staging)
 * the down launch also forms y: one workgroup computes all k instances of
 * its output rows and adds them in fp32, w[m][j] y_j from j = 0, rounding
 * once to binary16.  Otherwise each instance's output is rounded to
 * binary16 and a combine launch adds them in the same order.
 * ws/ws_bytes: at least qmlp_moe_workspace_bytes(...): a 1024-byte control
 * block (uint32 words on 128-byte lines: word 0 counts the calls and tags
 * each call's t words, word 160 holds sticky error bits, 1 = a wait for t
 * gave up), t as tagged 64-bit words [M*k][2r], h and the per-instance
 * outputs.  The workspace must be ZERO before its first call, and zeroed
 * again after a call failed or an error bit appeared (the results of that
 * call are invalid).  One workspace serves one call at a time: calls that
 * overlap in time on the same workspace race.
 */
size_t qmlp_moe_workspace_bytes(const qmlp_mlp *experts, int E, int M, int k, qmlp_dtype dtype);

qmlp_status qmlp_forward_moe(const qmlp_mlp *experts, int E, const void *x, int M,
                             qmlp_dtype dtype, const int32_t *topk_idx, const float *topk_w, int k,
                             void *y, void *ws, size_t ws_bytes, qmlp_stream stream);

/* Launch shape of qmlp_forward_moe's weight launches for M tokens with k
 * routed experts each (M k instances) of a [d][f] expert, on a device with
 * `cus` compute units: the lanes per row of the gate/up launch (gu_bits 2 or
 * 4) and of the down launch (dn_bits 2 or 4).  Gate/up: a few instances
 * leave the chip with fewer than two workgroups per compute unit at the
 * usual choice, so the lanes per row double (more, shorter rows per
 * workgroup) until it has them.  Returns 2 when down also forms the routing
 * sum (k <= 4; the fewest lanes with at most three 16-byte units each),
 * 1 when it takes the pipelined kernel and a combine launch follows, 0 the
 * plain kernel; -1 for arguments outside d, f > 0 and multiples of 64,
 * M, k >= 1, M k <= 40, cus >= 1, non-null outputs.  Host-only. */
int qmlp_moe_lanes(int d, int f, int gu_bits, int dn_bits, int M, int k, int cus,
                   int *gu_lanes, int *dn_lanes);

/* ---------------------------------------------- inspection (not timed) */

/*
 * Unpack a packed matrix into canonical form: codes uint8 [n][k] and the
 * binary16 bits of scale and zero [n][k/g] (QDQ view, Sec. 6.3).
 */
qmlp_status qmlp_unpack(const qmlp_qweight *w, uint8_t *codes, uint16_t *scales,
                        uint16_t *zeros, qmlp_stream stream);

/* The dequantized weight scale * (q - zero), rounded once to binary16
 * (nearest-even; q == zero gives +0), [n][k] row-major. */
qmlp_status qmlp_dequant(const qmlp_qweight *w, uint16_t *w_f16, qmlp_stream stream);

/* Number of kernel launches qmlp_forward makes for this block at M tokens:
 * 1 when the whole layer runs as one fused kernel (the decode shapes it
 * covers), 2 or 3 when it runs as the LoRA-A, gate/up and down kernels in
 * stream order; a bfloat16 prefill chunk makes LoRA-A and its reduction
 * (with an adapter), gate/up, down, and, when down splits f into slices to
 * fill the chip (f a multiple of 128 and fewer than 512 token x row tiles),
 * the slices' reduction; 0 if the call would be rejected.  Host-only,
 * enqueues nothing. */
int qmlp_forward_launches(const qmlp_mlp *mlp, int M, qmlp_dtype dtype);

/* Measurement hook (not part of the MLP): read `bytes` of device memory at
 * `buf` once with 128-bit loads -- the non-temporal form the weight stream
 * uses when `nontemporal` is nonzero, plain loads otherwise -- and write one
 * XOR word per wave to out[0 .. 4*blocks).  Decode is bound by the rate of
 * loading weights (Sec. 1, Sec. 3.3); this kernel does nothing but load, so
 * its duration is the HBM read rate this GPU sustains, and its byte
 * counters against the known size calibrate the counters of the decode
 * kernels.  One launch of `blocks` 256-thread workgroups.  bytes % 16 == 0,
 * 1 <= blocks <= 65536, buf 16-byte aligned, out 4-byte aligned. */
qmlp_status qmlp_probe_stream_read(const void *buf, size_t bytes, uint32_t *out, int blocks,
                                   int nontemporal, qmlp_stream stream);

/* A static, human-readable name of a status code. */
const char *qmlp_status_string(qmlp_status s);

#ifdef __cplusplus
}
#endif

#endif /* QMLP_H */
