// Kernel argument blocks and launchers shared between the C-ABI layer and
// the kernel translation units of libqmlp (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qmlp.h"

namespace qmlp {

// The argument checks of qmlp_forward that precede its workspace checks
// (descriptor, M, dtype, x and y); QMLP_OK for M == 0.
qmlp_status forward_check(const qmlp_mlp* mlp, const void* x, int M, qmlp_dtype dtype, const void* y);

// Codes per unit of a row's code stream: 32 at 4 bits and 64 at 2 bits (one
// 16-byte load); at 3 bits 64 (16 bytes of the 2-bit plane and 8 bytes of
// the 1-bit plane).
constexpr int codes_per_unit(int bits) { return bits == 4 ? 32 : 64; }

struct GateUpArgs {
    const uint32_t* cg;      // gate codes [f][d/16] words
    const uint32_t* mg;      // gate meta  [f][d/g]  (scale | zero << 16)
    const uint32_t* cu;      // up codes
    const uint32_t* mu;      // up meta
    const uint16_t* Bg;      // [f][r] binary16
    const uint16_t* Bu;      // [f][r] binary16
    const float* t;          // [M][2r] fp32: A_g x then A_u x
    const uint16_t* x;       // [M][d] binary16
    uint16_t* h;             // [M][f] binary16
    int M, d, f, g, r;
    int uc;                  // units per LDS chunk (set by the launcher)
    float lora_scale;
    int bits;                // code width of gate and up: 2, or 4 (uniform-W4 baseline)
};

struct DownArgs {
    const uint32_t* cd;      // down codes [d][f/8] words
    const uint32_t* md;      // down meta  [d][f/g]
    const uint16_t* h;       // [M][f] binary16
    uint16_t* y;             // [M][d] binary16
    int M, d, f, g;
    int uc;
    int bits;                // code width of down: 4, or 2 (uniform-W2 baseline)
};

hipError_t launch_pack(int bits, const float* W, int n, int k, int g, uint32_t* codes,
                       uint32_t* meta, int32_t* status, hipStream_t st);
hipError_t launch_unpack(int bits, const uint32_t* codes, const uint32_t* meta, int n, int k,
                         int g, uint8_t* out_codes, uint16_t* scales, uint16_t* zeros,
                         hipStream_t st);
hipError_t launch_dequant(int bits, const uint32_t* codes, const uint32_t* meta, int n, int k,
                          int g, uint16_t* out, hipStream_t st);

hipError_t launch_lora_a(const uint16_t* Ag, const uint16_t* Au, const uint16_t* x, int M, int d,
                         int r, float* t, hipStream_t st);
hipError_t launch_gateup(GateUpArgs args, hipStream_t st);
hipError_t launch_down(DownArgs args, hipStream_t st);
bool decode_shape_supported(int d, int f);
// Stand-alone decode kernels at gate/up code width bg with group gg and down
// code width bd (bg, bd in {2, 4}; group 32 only for gate/up, at either width,
// and for down at 4 bits).
bool decode_variant_supported(int d, int f, int bg, int gg, int bd, int gd);

// One kernel per layer (decode_fused.hip).  ctl: the 1 KB control block at
// the start of the workspace (zero before the first call); t64 [grid][256]
// and h32 [4][f]: the tagged hand-off words (zero before the first call).
bool fused_supported(int M, int d, int f, int g, int r);
int fused_grid();                              // blocks of the one-kernel layer (CU count)
hipError_t launch_fused(GateUpArgs gu, DownArgs dn, const uint16_t* Ag, const uint16_t* Au,
                        unsigned long long* t64, uint32_t* h32, unsigned* ctl, hipStream_t st);

// Prefill-chunk path (prefill.hip): M a multiple of 128 tokens, bfloat16.
bool prefill_supported(int M, int d, int f, int g, int r);
int prefill_splits(int d);
hipError_t launch_prefill_lora(const uint16_t* Ag, const uint16_t* Au, const uint16_t* x, int M,
                               int d, int r, float lora_scale, float* part, uint16_t* T,
                               hipStream_t st);
hipError_t launch_prefill_gateup(const uint32_t* cg, const uint32_t* mg, const uint32_t* cu,
                                 const uint32_t* mu, const uint16_t* x, const uint16_t* T,
                                 const uint16_t* Bg, const uint16_t* Bu, uint16_t* h, int M, int d,
                                 int f, int g, int r, hipStream_t st);
// Down over the chunk; with part (fp32 scratch of prefill_down_part_bytes)
// f is split into slices whose partial sums a second launch adds in slice
// order, else one launch writes y.
int prefill_down_slices(int M, int d, int f);
size_t prefill_down_part_bytes(int M, int d, int f);
hipError_t launch_prefill_down(const uint32_t* cd, const uint32_t* md, const uint16_t* h,
                               uint16_t* y, int M, int d, int f, int g, float* part, hipStream_t st);

// A stack of decode blocks in one persistent launch per up to
// stack_max_layers() layers (decode_stack.hip): M = 1, binary16, block l
// reads RMSNorm(x_l) and x_{l+1} = x_l + y_l.  ws: the stack area (stack_ws_bytes, zero before
// the first call).  launch_residual: out = x + y (binary16 or bfloat16).
struct StackLayerDesc {
    const uint32_t *cg, *mg, *cu, *mu, *cd, *md;
    const uint16_t *Bg, *Bu, *Ag, *Au;
    float lora_scale;
};
bool stack_supported(int M, int d, int f, int g, int r);

// A batch of up to kBatchMax independent decode blocks of one shape for the
// stand-alone kernels (blockIdx.y = block l): block l's weights come from
// lay[l], its activations sit at offset l of the batch buffers: x and y
// [nb][M][d], h [nb][M][f], t [nb][M][2r].  A single block is a batch of one.
constexpr int kBatchMax = 40;
struct BatchArgs {
    StackLayerDesc lay[kBatchMax];
    const uint16_t* x;
    uint16_t* y;
    uint16_t* h;
    float* t;
    int M, d, f, r;
    int gg, bg;              // gate/up group and code width
    int gd, bd;              // down group and code width
    int uc;                  // units per LDS chunk (set by the launcher)
    // Routed batches (mixture of experts): instance l runs the weights of
    // expert route[l] (a device array; 0 <= route[l] < nexp, clamped) on input
    // row group l / xdiv of x.  route == nullptr: instance l runs lay[l] on
    // x + l*M*d (xdiv 0 or 1).
    const int32_t* route;
    int nexp;
    int xdiv;
};
hipError_t launch_lora_a_batch(const BatchArgs& b, int nb, hipStream_t st);
// The routed-expert layer's control words (uint32 indices into the
// workspace's control block, each on its own 128-byte line): the call
// counter, whose value plus one tags this call's LoRA-A words, and sticky
// error bits (1 = a wait for t gave up).
constexpr int kMoeCtlEpoch = 0, kMoeCtlErr = 160;
// Gate/up over a routed batch at one token with the LoRA-A projection in the
// same launch: the first workgroups of each instance compute t and publish
// it as tagged 64-bit words (fp32 bits | tag << 32) in t64 [nb][2r]; the
// gate/up workgroups read them for the LoRA-B term.  gateup_routed_fits says
// whether it takes the shape (rank > 0, one token per instance).
bool gateup_routed_fits(const BatchArgs& b, int nb);
hipError_t launch_gateup_routed_batch(const BatchArgs& b, int nb, unsigned long long* t64, unsigned* ctl,
                                    hipStream_t st);
// Down over a routed batch (M = 1, k = xdiv instances per token) with the
// routing-weighted combine folded in: y [nb/k][d] binary16, w [nb/k][k].
// down_combine_fits says whether the folded kernel takes the shape (k <= 4,
// the instances' h within its staging); otherwise launch_down_combine
// returns hipErrorInvalidValue before launching anything.
bool down_combine_fits(const BatchArgs& b, int nb);
// ctl: the control block; its call counter advances once the sums are written.
hipError_t launch_down_combine(const BatchArgs& b, int nb, const float* w, uint16_t* y, unsigned* ctl,
                               hipStream_t st);
// The streamed path of a batch at one token (decode_stream.hip): one
// persistent gate/up launch (with LoRA-A) and one persistent down launch
// over all blocks of the batch.  Binary16, 2-bit gate/up and 4-bit
// down at groups 64/128, rank 0/8/16/32, d % 512 == 0, d <= 4096,
// f % 128 == 0, f <= 12288 (plus the LDS and span limits it checks).
bool stream_supported(int M, int d, int f, int gg, int bg, int gd, int bd, int r, int nb);
// With adapters the gate/up launch also computes LoRA-A (extra workgroups
// after the streaming ones) and hands t over as tagged words in t64
// [nb][2r] (fp32 | tag << 32); the tag is the call counter in ctl (word 0)
// plus one, which the down launch advances; word 160 holds sticky error
// bits (1 = a wait for t gave up).
hipError_t launch_gateup_stream(const BatchArgs& b, int nb, unsigned long long* t64, unsigned* ctl,
                                hipStream_t st);
hipError_t launch_down_stream(const BatchArgs& b, int nb, unsigned* ctl, hipStream_t st);
// The matrix-core path of a batch at 3..16 tokens (decode_mfma.hip): one
// persistent gate/up launch and one persistent down launch over all blocks
// of the batch, after launch_lora_a_mfma.  Binary16, 2-bit gate/up and
// 4-bit down at groups 64/128, rank 0/8/16/32, d % 512 == 0,
// f % 256 == 0 (plus the LDS limits it checks).
bool mfma_supported(int M, int d, int f, int gg, int bg, int gd, int bd, int r, int nb);
// Its LoRA-A products t = [A_g; A_u] x (r > 0) as fp32 partial sums over
// kLoraSlices slices of d, t [kLoraSlices][nb][M][2r]; the gate/up launch
// adds them in slice order.
constexpr int kLoraSlices = 4;
hipError_t launch_lora_a_mfma(const BatchArgs& b, int nb, hipStream_t st);
hipError_t launch_gateup_mfma(const BatchArgs& b, int nb, hipStream_t st);
hipError_t launch_down_mfma(const BatchArgs& b, int nb, hipStream_t st);
hipError_t launch_gateup_batch(const BatchArgs& b, int nb, hipStream_t st);
hipError_t launch_down_batch(const BatchArgs& b, int nb, hipStream_t st);
// y[m] = sum_j w[m k + j] * yi[m k + j] over the k routed experts of token m
// (fp32 sum, one rounding to binary16); yi [M k][d], w [M k], y [M][d].
// ctl (may be null): the routed layer's control block, whose call counter
// advances.
hipError_t launch_moe_combine(const uint16_t* yi, const float* w, int M, int k, int d, uint16_t* y,
                              unsigned* ctl, hipStream_t st);
size_t stack_ws_bytes(int d, int f, int r);
int stack_max_layers();
// Byte offset of the persistent stack launch's sticky error word in its area.
size_t stack_error_word_offset();
hipError_t launch_stack(const StackLayerDesc* layers, int L, int d, int f, int g, int r,
                        const uint16_t* x0, uint16_t* y, uint16_t* x_last, void* ws, hipStream_t st);
hipError_t launch_residual(const uint16_t* x, const uint16_t* y, uint16_t* out, int n, bool bf16,
                           hipStream_t st);
hipError_t launch_rmsnorm(const uint16_t* x, uint16_t* u, int M, int d, hipStream_t st);

}  // namespace qmlp
