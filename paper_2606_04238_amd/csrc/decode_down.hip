// Stand-alone decode kernel of the down projection y = Wdown h: 4-bit
// (Sec. 3.3), or 2-bit for the uniform-W2 baseline of the precision
// comparison (Sec. 5.2); serves qmlp_down_w4, the shapes and widths the
// fused layer kernel does not cover, and batches of independent blocks
// (blockIdx.y = block).
#include "decode_standalone.h"

namespace qmlp {

QMLP_SA_EXTERN

// Launch shape of the down kernel.  Every block stages all of h (M tokens
// of f) for a few rows, so batches take the fewest lanes per row (more rows
// per block) and, at M >= 2 tokens, 1024-thread blocks; single blocks keep
// 256 threads and the lanes of lanes_for (more blocks to fill the chip).
// Measured on batches of Qwen3-4B blocks at one token (W4 and W2 down) and
// Qwen3-8B blocks at 4 and 16 tokens.
static bool down_big_blocks(int nb, int M) { return nb > 1 && M > 1; }

hipError_t launch_down_batch(const BatchArgs& b, int nb, hipStream_t st) {
    if (nb < 1 || nb > kBatchMax)
        return hipErrorInvalidValue;
    const bool big = down_big_blocks(nb, b.M);
    const int U = b.f / codes_per_unit(b.bd);
    const int S = nb > 1 ? lanes_fewest(U) : lanes_for(U, b.bd);
    if (b.bd == 4)
        return big ? launch_down_bits<4, 1024>(b, nb, S, st) : launch_down_bits<4, 256>(b, nb, S, st);
    if (b.bd == 2 && b.gd != 32)
        return big ? launch_down_bits<2, 1024>(b, nb, S, st) : launch_down_bits<2, 256>(b, nb, S, st);
    return hipErrorInvalidValue;
}

}  // namespace qmlp

extern "C" int qmlp_moe_lanes(int d, int f, int gu_bits, int dn_bits, int M, int k, int cus, int* gu_lanes,
                              int* dn_lanes) {
    using namespace qmlp;
    const int instances = M * k;
    if (d <= 0 || f <= 0 || M < 1 || k < 1 || instances > kBatchMax || cus < 1 || !gu_lanes || !dn_lanes ||
        (gu_bits != 2 && gu_bits != 4) || (dn_bits != 2 && dn_bits != 4) || d % 64 != 0 || f % 64 != 0)
        return -1;
    *gu_lanes = routed_gateup_lanes(d / codes_per_unit(gu_bits), f, instances, gu_bits, cus);
    const int Ud = f / codes_per_unit(dn_bits);
    if (down_combine_fits_shape(d, f, k, dn_bits)) {
        *dn_lanes = combine_lanes(Ud);
        return 2;
    }
    const bool pipe = down_pipe_fits_shape(d, f, 1, instances, dn_bits);
    *dn_lanes = pipe ? routed_pipe_lanes(Ud, d, instances, cus) : instances > 1 ? lanes_fewest(Ud) : lanes_for(Ud, dn_bits);
    return pipe ? 1 : 0;
}

namespace qmlp {

// One thread per output element: the routing-weighted sum of the k expert
// outputs of its token (Sec. 5 names the routed experts of the MoE decoder;
// the weights come with the routing).  KM >= k: every load of a thread is
// issued before the first add (the slots past k re-read slot k - 1 and are
// dropped), so the kernel makes one trip to memory; the sum runs over
// j = 0 .. k - 1 in order.
template <int KM>
__global__ void __launch_bounds__(256)
moe_combine_kernel(const uint16_t* __restrict__ yi, const float* __restrict__ w, int M, int k,
                   int d, uint16_t* __restrict__ y, unsigned* ctl) {
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0 && ctl)
        advance_call_counter(ctl + kMoeCtlEpoch);
    if (i >= (long)M * d)
        return;
    const long m = i / d, c = i - m * d;
    float wv[KM];
    uint32_t yv[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
        const int jj = j < k ? j : k - 1;
        wv[j] = w[m * k + jj];
        yv[j] = yi[(m * k + jj) * d + c];
    }
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < KM; ++j)
        if (j < k)
            acc += wv[j] * h2f(yv[j]);
    y[i] = (uint16_t)f2h(acc);
}

hipError_t launch_moe_combine(const uint16_t* yi, const float* w, int M, int k, int d, uint16_t* y,
                              unsigned* ctl, hipStream_t st) {
    const long n = (long)M * d;
    const unsigned grid = (unsigned)((n + 255) / 256);
    if (k <= 4)
        moe_combine_kernel<4><<<grid, 256, 0, st>>>(yi, w, M, k, d, y, ctl);
    else if (k <= 8)
        moe_combine_kernel<8><<<grid, 256, 0, st>>>(yi, w, M, k, d, y, ctl);
    else
        moe_combine_kernel<kBatchMax><<<grid, 256, 0, st>>>(yi, w, M, k, d, y, ctl);
    return hipGetLastError();
}

bool down_combine_fits(const BatchArgs& b, int nb) {
    return b.route && b.M == 1 && b.xdiv >= 1 && nb % b.xdiv == 0 && (b.bd == 4 || (b.bd == 2 && b.gd != 32)) &&
           down_combine_fits_shape(b.d, b.f, b.xdiv, b.bd);
}

hipError_t launch_down_combine(const BatchArgs& b, int nb, const float* w, uint16_t* y, unsigned* ctl,
                               hipStream_t st) {
    if (nb < 1 || nb > kBatchMax || !w || !y || !down_combine_fits(b, nb))
        return hipErrorInvalidValue;
    return b.bd == 4 ? launch_down_pipe_combine<4>(b, nb, w, y, ctl, st)
                     : launch_down_pipe_combine<2>(b, nb, w, y, ctl, st);
}

// A single block as a batch of one.
hipError_t launch_down(DownArgs a, hipStream_t st) {
    BatchArgs b{};
    b.lay[0].cd = a.cd;
    b.lay[0].md = a.md;
    b.h = const_cast<uint16_t*>(a.h);
    b.y = a.y;
    b.M = a.M;
    b.d = a.d;
    b.f = a.f;
    b.gd = a.g;
    b.bd = a.bits;
    return launch_down_batch(b, 1, st);
}

}  // namespace qmlp
