// Stand-alone decode kernels of the gate/up half: the LoRA-A projection
// t = [A_g; A_u] x and the fused gate/up dequant-matvec with the LoRA-B term
// and the SiLU(G) * U epilogue (Sec. 3.1 Eq. (1), Sec. 3.3, Sec. 4.2,
// Sec. 5).  qmlp_forward normally runs the single fused layer kernel instead
// (decode_fused.hip); these serve qmlp_gateup_w2_lora, the shapes and code
// widths the fused kernel does not cover, and batches of independent blocks
// (blockIdx.y = block), a single block being a batch of one.
#include "decode_standalone.h"

namespace qmlp {

QMLP_SA_EXTERN

// One wave per row c of [A_g; A_u] of block blockIdx.y.
template <int MT>
__global__ void __launch_bounds__(256)
lora_a_kernel(BatchArgs b) {
    const int l = blockIdx.y;
    const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (wave >= 2 * b.r)
        return;
    const int e = batch_expert(b, l);
    lora_a_row<MT, (MT <= 4 ? 12 / MT : 1)>(b.lay[e].Ag, b.lay[e].Au, batch_x(b, l), b.M, b.d,
                                            b.r, wave, b.t + (long)l * b.M * 2 * b.r,
                                            threadIdx.x & 63);
}

hipError_t launch_lora_a_batch(const BatchArgs& b, int nb, hipStream_t st) {
    const dim3 grid((unsigned)((2 * b.r * 64 + 255) / 256), (unsigned)nb);
    switch (mtile_for(b.M)) {
    case 1: lora_a_kernel<1><<<grid, 256, 0, st>>>(b); break;
    case 2: lora_a_kernel<2><<<grid, 256, 0, st>>>(b); break;
    case 4: lora_a_kernel<4><<<grid, 256, 0, st>>>(b); break;
    case 8: lora_a_kernel<8><<<grid, 256, 0, st>>>(b); break;
    default: lora_a_kernel<16><<<grid, 256, 0, st>>>(b); break;
    }
    return hipGetLastError();
}

// Launch shape of the gate/up kernel: 256-thread blocks with the lanes of
// lanes_for, single blocks and batches alike (a sweep of 1024-thread blocks
// and of the fewest lanes per row over the Qwen3-4B widths at one token
// and the Qwen3-8B block at 4 and 16 tokens found nothing faster: x is a
// small share of a block's bytes).
hipError_t launch_gateup_batch(const BatchArgs& b, int nb, hipStream_t st) {
    if (nb < 1 || nb > kBatchMax)
        return hipErrorInvalidValue;
    const int U = b.d / codes_per_unit(b.bg);
    // A routed launch over a few expert instances (one token, top-k) leaves
    // the chip with fewer than two workgroups per CU at lanes_for's choice:
    // routed_gateup_lanes doubles the lanes per row until it has them.
    // GPT-OSS-20B-class experts, 2-bit gate/up, top-4: 8 -> 16 lanes,
    // 360 -> 720 workgroups, 31.3 -> 27.7 us per MoE layer.
    const int S = b.route ? routed_gateup_lanes(U, b.f, nb, b.bg, device_cu_count()) : lanes_for(U, b.bg);
    if (b.bg == 4)
        return launch_gateup_bits<4, false, 256>(b, nb, S, st);
    if (b.bg == 3)
        return b.gg == 32 ? launch_gateup_bits<3, true, 256>(b, nb, S, st)
                          : launch_gateup_bits<3, false, 256>(b, nb, S, st);
    if (b.bg == 2 && b.gg == 32)
        return launch_gateup_bits<2, true, 256>(b, nb, S, st);
    if (b.bg == 2)
        return launch_gateup_bits<2, false, 256>(b, nb, S, st);
    return hipErrorInvalidValue;
}

bool gateup_routed_fits(const BatchArgs& b, int nb) {
    return nb >= 1 && nb <= kBatchMax && b.M == 1 && b.r >= 0 && 2 * b.r <= 64 &&
           (b.bg == 2 || b.bg == 3 || b.bg == 4);
}

// The lanes per row are those of launch_gateup_batch.
hipError_t launch_gateup_routed_batch(const BatchArgs& b, int nb, unsigned long long* t64, unsigned* ctl,
                                    hipStream_t st) {
    if (!gateup_routed_fits(b, nb))
        return hipErrorInvalidValue;
    const int U = b.d / codes_per_unit(b.bg);
    const int S = b.route ? routed_gateup_lanes(U, b.f, nb, b.bg, device_cu_count()) : lanes_for(U, b.bg);
    if (b.bg == 4)
        return launch_gateup_routed_bits<4, false>(b, nb, S, t64, ctl, st);
    if (b.bg == 3)
        return b.gg == 32 ? launch_gateup_routed_bits<3, true>(b, nb, S, t64, ctl, st)
                          : launch_gateup_routed_bits<3, false>(b, nb, S, t64, ctl, st);
    return b.gg == 32 ? launch_gateup_routed_bits<2, true>(b, nb, S, t64, ctl, st)
                      : launch_gateup_routed_bits<2, false>(b, nb, S, t64, ctl, st);
}

// A single block as a batch of one.
static BatchArgs single_gateup(const GateUpArgs& a) {
    BatchArgs b{};
    StackLayerDesc& w = b.lay[0];
    w.cg = a.cg;
    w.mg = a.mg;
    w.cu = a.cu;
    w.mu = a.mu;
    w.Bg = a.Bg;
    w.Bu = a.Bu;
    w.lora_scale = a.lora_scale;
    b.x = a.x;
    b.h = a.h;
    b.t = const_cast<float*>(a.t);
    b.M = a.M;
    b.d = a.d;
    b.f = a.f;
    b.r = a.r;
    b.gg = a.g;
    b.bg = a.bits;
    return b;
}

hipError_t launch_lora_a(const uint16_t* Ag, const uint16_t* Au, const uint16_t* x, int M, int d,
                         int r, float* t, hipStream_t st) {
    BatchArgs b{};
    b.lay[0].Ag = Ag;
    b.lay[0].Au = Au;
    b.x = x;
    b.t = t;
    b.M = M;
    b.d = d;
    b.r = r;
    return launch_lora_a_batch(b, 1, st);
}

hipError_t launch_gateup(GateUpArgs args, hipStream_t st) {
    return launch_gateup_batch(single_gateup(args), 1, st);
}

bool decode_shape_supported(int d, int f) { return decode_shape_supported_impl(d, f); }

bool decode_variant_supported(int d, int f, int bg, int gg, int bd, int gd) {
    if ((bg != 2 && bg != 3 && bg != 4) || (bd != 2 && bd != 4))
        return false;
    if (gg != 32 && gg != 64 && gg != 128)
        return false;
    if ((gd != 32 && gd != 64 && gd != 128) || (bd == 2 && gd == 32))
        return false;
    return d % 64 == 0 && f % 64 == 0 && d % gg == 0 && f % gd == 0 && units_fit(d, bg) &&
           units_fit(f, bd);
}

}  // namespace qmlp
