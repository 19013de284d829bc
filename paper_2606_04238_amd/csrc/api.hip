// C ABI of libqmlp: argument validation, workspace layout and kernel dispatch.
// Every check runs before the first launch, so a rejected call enqueues
// nothing and writes nothing.
#include <cstring>
#include <stddef.h>
#include <stdint.h>

#include "qmlp.h"
#include "qmlp_internal.h"
#include "decode_launch.h"

namespace {

using namespace qmlp;

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

inline size_t round256(size_t v) { return (v + 255) & ~(size_t)255; }

qmlp_status from_hip(hipError_t e) { return e == hipSuccess ? QMLP_OK : QMLP_ERR_HIP; }

// Structural checks of one packed-weight view (bits 0 = either width).
qmlp_status check_qweight(const qmlp_qweight* w, int bits) {
    if (!w || !w->codes || !w->meta)
        return QMLP_ERR_NULL;
    if (bits ? w->bits != bits : (w->bits < 2 || w->bits > 4))
        return QMLP_ERR_UNSUPPORTED;
    if (w->n_out <= 0 || w->k_in <= 0)
        return QMLP_ERR_SHAPE;
    if (w->group != 32 && w->group != 64 && w->group != 128)
        return QMLP_ERR_UNSUPPORTED;
    if (w->k_in % w->group != 0 || (w->bits == 3 && w->k_in % 128 != 0))
        return QMLP_ERR_SHAPE;
    if (!aligned16(w->codes) || !aligned16(w->meta))
        return QMLP_ERR_ALIGN;
    return QMLP_OK;
}

// The W4/W2-GateUp block (2-bit gate/up, 4-bit down, groups of 64 or 128):
// the only form the fused, persistent and prefill kernels take.  The other
// widths (uniform W4, uniform W2) and group 32 -- the comparison points of
// Sec. 5.2 and the paper's own INT2 grouping -- run on the stand-alone
// decode kernels.
bool standard_mlp(const qmlp_mlp* mlp) {
    return mlp->gate.bits == 2 && mlp->down.bits == 4 && mlp->gate.group >= 64 &&
           mlp->down.group >= 64;
}

// Shape, pointer and type checks of a whole block at M tokens.
qmlp_status check_mlp(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    if (!mlp)
        return QMLP_ERR_NULL;
    qmlp_status s;
    if ((s = check_qweight(&mlp->gate, 0)) != QMLP_OK) return s;
    if ((s = check_qweight(&mlp->up, mlp->gate.bits)) != QMLP_OK) return s;
    if ((s = check_qweight(&mlp->down, 0)) != QMLP_OK) return s;
    const int f = mlp->gate.n_out, d = mlp->gate.k_in;
    if (mlp->up.n_out != f || mlp->up.k_in != d || mlp->down.n_out != d || mlp->down.k_in != f)
        return QMLP_ERR_SHAPE;
    if (mlp->up.group != mlp->gate.group)
        return QMLP_ERR_SHAPE;
    if ((mlp->down.bits == 2 && mlp->down.group == 32) || mlp->down.bits == 3)
        return QMLP_ERR_UNSUPPORTED;
    if (d % 64 != 0 || f % 64 != 0)
        return QMLP_ERR_SHAPE;
    if (mlp->rank != 0 && mlp->rank != 8 && mlp->rank != 16 && mlp->rank != 32)
        return QMLP_ERR_UNSUPPORTED;
    if (mlp->rank > 0) {
        if (!mlp->A_gate || !mlp->B_gate || !mlp->A_up || !mlp->B_up)
            return QMLP_ERR_NULL;
        if (!aligned16(mlp->A_gate) || !aligned16(mlp->B_gate) || !aligned16(mlp->A_up) ||
            !aligned16(mlp->B_up))
            return QMLP_ERR_ALIGN;
    }
    if (M < 0)
        return QMLP_ERR_SHAPE;
    if (dtype == QMLP_BF16) {                    // prefill-chunk path
        if (!standard_mlp(mlp) ||
            (M != 0 && !prefill_supported(M, d, f, mlp->gate.group, mlp->rank)))
            return QMLP_ERR_UNSUPPORTED;
        return QMLP_OK;
    }
    if (dtype != QMLP_F16)
        return QMLP_ERR_UNSUPPORTED;
    if (M > 16)                                  // decode runs in binary16 at 1..16 tokens
        return QMLP_ERR_UNSUPPORTED;
    if (!decode_shape_supported(d, f) ||
        !decode_variant_supported(d, f, mlp->gate.bits, mlp->gate.group, mlp->down.bits,
                                  mlp->down.group))
        return QMLP_ERR_UNSUPPORTED;
    return QMLP_OK;
}

// Workspace: [control words, 1 KB][t: fp32][h: M x f activation type]
// [T: M x 2r bfloat16, prefill only][t64: one [4][64] copy of tagged words
// per block of the one-kernel layer, h32: 4 x f tagged words -- decode only,
// that kernel's hand-offs].  t is
// M x 2r on the decode path and S x M x 2r split-K partials on the prefill
// path.
constexpr size_t kCtlBytes = 1024;

struct Workspace {
    unsigned* ctl;
    float* t;
    uint16_t* h;
    uint16_t* T;
    unsigned long long* t64;
    uint32_t* h32;
    float* part;                // prefill down partial sums (bfloat16 chunks), else null
};

size_t ws_t_bytes(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    const size_t S = dtype == QMLP_BF16 ? (size_t)prefill_splits(mlp->gate.k_in) : 1;
    return round256(S * (size_t)M * 2 * mlp->rank * 4);
}
size_t ws_h_bytes(const qmlp_mlp* mlp, int M) { return round256((size_t)M * mlp->gate.n_out * 2); }
size_t ws_T_bytes(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    return dtype == QMLP_BF16 ? round256((size_t)M * 2 * mlp->rank * 2) : 0;
}
size_t ws_t64_bytes() { return (size_t)fused_grid() * 256 * 8; }
size_t ws_tag_bytes(const qmlp_mlp* mlp, qmlp_dtype dtype) {
    return dtype == QMLP_F16 ? ws_t64_bytes() + round256((size_t)4 * mlp->gate.n_out * 4) : 0;
}
size_t ws_part_bytes(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    return dtype == QMLP_BF16 ? round256(prefill_down_part_bytes(M, mlp->gate.k_in, mlp->gate.n_out)) : 0;
}
// Everything qmlp_forward carves from its workspace.
size_t ws_total_bytes(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    return kCtlBytes + ws_t_bytes(mlp, M, dtype) + ws_h_bytes(mlp, M) + ws_T_bytes(mlp, M, dtype) +
           ws_tag_bytes(mlp, dtype) + ws_part_bytes(mlp, M, dtype);
}

Workspace carve(const qmlp_mlp* mlp, int M, qmlp_dtype dtype, void* ws) {
    char* base = static_cast<char*>(ws);
    const size_t tb = ws_t_bytes(mlp, M, dtype), hb = ws_h_bytes(mlp, M);
    char* tag = base + kCtlBytes + tb + hb + ws_T_bytes(mlp, M, dtype);
    char* part = tag + ws_tag_bytes(mlp, dtype);
    return {reinterpret_cast<unsigned*>(base), reinterpret_cast<float*>(base + kCtlBytes),
            reinterpret_cast<uint16_t*>(base + kCtlBytes + tb),
            reinterpret_cast<uint16_t*>(base + kCtlBytes + tb + hb),
            reinterpret_cast<unsigned long long*>(tag),
            reinterpret_cast<uint32_t*>(tag + (dtype == QMLP_F16 ? ws_t64_bytes() : 0)),
            ws_part_bytes(mlp, M, dtype) ? reinterpret_cast<float*>(part) : nullptr};
}

// The prefill-chunk gate/up half: LoRA-A (split K + reduction), then the
// MFMA gate/up kernel with the LoRA products and SiLU(G) * U.
qmlp_status run_prefill_gateup(const qmlp_mlp* mlp, const void* x, int M, uint16_t* h,
                               const Workspace& w, hipStream_t st) {
    const int d = mlp->gate.k_in, f = mlp->gate.n_out, r = mlp->rank;
    if (r > 0) {
        hipError_t e = launch_prefill_lora(static_cast<const uint16_t*>(mlp->A_gate),
                                           static_cast<const uint16_t*>(mlp->A_up),
                                           static_cast<const uint16_t*>(x), M, d, r,
                                           mlp->lora_scale, w.t, w.T, st);
        if (e != hipSuccess)
            return QMLP_ERR_HIP;
    }
    return from_hip(launch_prefill_gateup(
        static_cast<const uint32_t*>(mlp->gate.codes), static_cast<const uint32_t*>(mlp->gate.meta),
        static_cast<const uint32_t*>(mlp->up.codes), static_cast<const uint32_t*>(mlp->up.meta),
        static_cast<const uint16_t*>(x), w.T, static_cast<const uint16_t*>(mlp->B_gate),
        static_cast<const uint16_t*>(mlp->B_up), h, M, d, f, mlp->gate.group, r, st));
}

qmlp_status run_prefill_down(const qmlp_qweight* down, const void* h, int M, void* y, float* part,
                             hipStream_t st) {
    return from_hip(launch_prefill_down(static_cast<const uint32_t*>(down->codes),
                                        static_cast<const uint32_t*>(down->meta),
                                        static_cast<const uint16_t*>(h), static_cast<uint16_t*>(y),
                                        M, down->n_out, down->k_in, down->group, part, st));
}

GateUpArgs gateup_args(const qmlp_mlp* mlp, const void* x, int M, uint16_t* h, const float* t) {
    GateUpArgs a;
    a.cg = static_cast<const uint32_t*>(mlp->gate.codes);
    a.mg = static_cast<const uint32_t*>(mlp->gate.meta);
    a.cu = static_cast<const uint32_t*>(mlp->up.codes);
    a.mu = static_cast<const uint32_t*>(mlp->up.meta);
    // With rank 0 the kernels still issue (unused) loads of the LoRA-B
    // slices; point them at x, which is always readable.
    a.Bg = static_cast<const uint16_t*>(mlp->rank > 0 ? mlp->B_gate : x);
    a.Bu = static_cast<const uint16_t*>(mlp->rank > 0 ? mlp->B_up : x);
    a.t = t;
    a.x = static_cast<const uint16_t*>(x);
    a.h = h;
    a.M = M;
    a.d = mlp->gate.k_in;
    a.f = mlp->gate.n_out;
    a.g = mlp->gate.group;
    a.r = mlp->rank;
    a.uc = 0;
    a.lora_scale = mlp->lora_scale;
    a.bits = mlp->gate.bits;
    return a;
}

DownArgs down_args(const qmlp_qweight* down, const void* h, int M, void* y) {
    DownArgs a;
    a.cd = static_cast<const uint32_t*>(down->codes);
    a.md = static_cast<const uint32_t*>(down->meta);
    a.h = static_cast<const uint16_t*>(h);
    a.y = static_cast<uint16_t*>(y);
    a.M = M;
    a.d = down->n_out;
    a.f = down->k_in;
    a.g = down->group;
    a.uc = 0;
    a.bits = down->bits;
    return a;
}

// The gate/up half: LoRA-A projection then the fused kernel.
qmlp_status run_gateup(const qmlp_mlp* mlp, const void* x, int M, uint16_t* h, float* t,
                       hipStream_t st) {
    if (mlp->rank > 0) {
        hipError_t e = launch_lora_a(static_cast<const uint16_t*>(mlp->A_gate),
                                     static_cast<const uint16_t*>(mlp->A_up),
                                     static_cast<const uint16_t*>(x), M, mlp->gate.k_in,
                                     mlp->rank, t, st);
        if (e != hipSuccess)
            return QMLP_ERR_HIP;
    }
    return from_hip(launch_gateup(gateup_args(mlp, x, M, h, t), st));
}

qmlp_status pack_common(int bits, const float* W, int n_out, int k_in, int group,
                        qmlp_qweight* out, int32_t* d_status, qmlp_stream stream) {
    if (!W || !out || !out->codes || !out->meta)
        return QMLP_ERR_NULL;
    if (n_out <= 0 || k_in <= 0)
        return QMLP_ERR_SHAPE;
    if (group != 32 && group != 64 && group != 128)
        return QMLP_ERR_UNSUPPORTED;
    if (k_in % group != 0 || (bits == 3 && k_in % 128 != 0))
        return QMLP_ERR_SHAPE;
    if (!aligned16(W) || !aligned16(out->codes) || !aligned16(out->meta))
        return QMLP_ERR_ALIGN;
    if (d_status && ((uintptr_t)d_status & 3u))
        return QMLP_ERR_ALIGN;
    hipError_t e = launch_pack(bits, W, n_out, k_in, group, static_cast<uint32_t*>(out->codes),
                               static_cast<uint32_t*>(out->meta), d_status,
                               static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return QMLP_ERR_HIP;
    out->bits = bits;
    out->n_out = n_out;
    out->k_in = k_in;
    out->group = group;
    return QMLP_OK;
}

qmlp_status check_inspect(const qmlp_qweight* w) {
    if (!w)
        return QMLP_ERR_NULL;
    return check_qweight(w, 0);
}

// L independent blocks of one shape: block l maps x[l] to y[l].
qmlp_status check_layers(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (!layers)
        return QMLP_ERR_NULL;
    if (L <= 0)
        return QMLP_ERR_SHAPE;
    for (int i = 0; i < L; ++i) {
        qmlp_status s = check_mlp(&layers[i], M, dtype);
        if (s != QMLP_OK)
            return s;
        const qmlp_mlp& a = layers[0];
        const qmlp_mlp& b = layers[i];
        if (b.gate.k_in != a.gate.k_in || b.gate.n_out != a.gate.n_out || b.gate.group != a.gate.group ||
            b.down.group != a.down.group || b.rank != a.rank || b.gate.bits != a.gate.bits ||
            b.down.bits != a.down.bits)
            return QMLP_ERR_SHAPE;
    }
    return QMLP_OK;
}

// A stack of blocks of one shape: layer l+1's input is layer l's output.
qmlp_status check_stack(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    const qmlp_status s = check_layers(layers, L, M, dtype);
    if (s != QMLP_OK)
        return s;
    return dtype == QMLP_F16 ? QMLP_OK : QMLP_ERR_UNSUPPORTED;   // the stream and the norm are binary16
}

bool stack_persistent(const qmlp_mlp* layers, int M, qmlp_dtype dtype) {
    const qmlp_mlp& a = layers[0];
    return dtype == QMLP_F16 && standard_mlp(&a) && a.down.group == a.gate.group &&
           stack_supported(M, a.gate.k_in, a.gate.n_out, a.gate.group, a.rank);
}

size_t stack_layer_ws(const qmlp_mlp* layers, int M, qmlp_dtype dtype) {
    return round256(ws_total_bytes(layers, M, dtype));
}

StackLayerDesc stack_desc(const qmlp_mlp& m) {
    StackLayerDesc s;
    s.cg = static_cast<const uint32_t*>(m.gate.codes);
    s.mg = static_cast<const uint32_t*>(m.gate.meta);
    s.cu = static_cast<const uint32_t*>(m.up.codes);
    s.mu = static_cast<const uint32_t*>(m.up.meta);
    s.cd = static_cast<const uint32_t*>(m.down.codes);
    s.md = static_cast<const uint32_t*>(m.down.meta);
    s.Bg = static_cast<const uint16_t*>(m.B_gate);
    s.Bu = static_cast<const uint16_t*>(m.B_up);
    s.Ag = static_cast<const uint16_t*>(m.A_gate);
    s.Au = static_cast<const uint16_t*>(m.A_up);
    s.lora_scale = m.lora_scale;
    return s;
}

// Independent blocks at one token in the W4/W2-GateUp form stream: every
// batch of up to kBatchMax blocks is the LoRA-A launch, one persistent
// gate/up launch and one persistent down launch (decode_stream.hip).
bool layers_streamed(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    const qmlp_mlp& a = layers[0];
    if (dtype != QMLP_F16 || !standard_mlp(&a))
        return false;
    const int full = L / kBatchMax, rest = L % kBatchMax;
    const auto ok = [&](int nb) {
        return stream_supported(M, a.gate.k_in, a.gate.n_out, a.gate.group, a.gate.bits, a.down.group,
                                a.down.bits, a.rank, nb);
    };
    return (full == 0 || ok(kBatchMax)) && (rest == 0 || ok(rest));
}

// Independent blocks at 3..16 tokens in the W4/W2-GateUp form run on the
// matrix cores: every batch is the LoRA-A launch, one persistent gate/up
// launch and one persistent down launch (decode_mfma.hip).
bool layers_mfma(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    const qmlp_mlp& a = layers[0];
    if (dtype != QMLP_F16 || !standard_mlp(&a))
        return false;
    const int full = L / kBatchMax, rest = L % kBatchMax;
    const auto ok = [&](int nb) {
        return mfma_supported(M, a.gate.k_in, a.gate.n_out, a.gate.group, a.gate.bits, a.down.group,
                              a.down.bits, a.rank, nb);
    };
    return (full == 0 || ok(kBatchMax)) && (rest == 0 || ok(rest));
}

// Independent blocks that neither stream nor take the matrix cores run in
// batches of up to kBatchMax blocks on the stand-alone kernels: LoRA-A of
// every block of the batch, then gate/up of every block, then down of every
// block (three launches per batch, two without adapters).  Binary16 decode
// only; bfloat16 runs qmlp_forward per block.
bool layers_batched(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    return dtype == QMLP_F16 && !layers_streamed(layers, L, M, dtype) && !layers_mfma(layers, L, M, dtype);
}

enum class BatchPath { kBatched, kStreamed, kMfma };

BatchPath batch_path(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    return layers_streamed(layers, L, M, dtype) ? BatchPath::kStreamed
           : layers_mfma(layers, L, M, dtype)   ? BatchPath::kMfma
                                                : BatchPath::kBatched;
}

// t of a batch: [nb][M][2r] fp32, or kLoraSlices such arrays of partial
// sums on the matrix-core path.
size_t batch_t_bytes(const qmlp_mlp* a, int nb, int M, int slices = 1) {
    return round256((size_t)slices * nb * M * 2 * a->rank * 4);
}
size_t batch_h_bytes(const qmlp_mlp* a, int nb, int M) {
    return round256((size_t)nb * M * a->gate.n_out * 2);
}
int batch_size(int L) { return L < kBatchMax ? L : kBatchMax; }

qmlp_status run_layers_batched(const qmlp_mlp* layers, int L, const char* xb, int M, char* yb,
                               void* ws, hipStream_t st, BatchPath path) {
    const qmlp_mlp& a = layers[0];
    const int d = a.gate.k_in;
    const size_t step = (size_t)M * d * 2;
    char* base = static_cast<char*>(ws);
    // t: four fp32 partial sums per value on the matrix cores, one tagged
    // 64-bit word on the streamed path, fp32 otherwise
    const int ts = path == BatchPath::kMfma ? kLoraSlices : path == BatchPath::kStreamed ? 2 : 1;
    BatchArgs b{};
    b.t = reinterpret_cast<float*>(base + kCtlBytes);
    b.h = reinterpret_cast<uint16_t*>(base + kCtlBytes + batch_t_bytes(&a, batch_size(L), M, ts));
    b.M = M;
    b.d = d;
    b.f = a.gate.n_out;
    b.r = a.rank;
    b.gg = a.gate.group;
    b.bg = a.gate.bits;
    b.gd = a.down.group;
    b.bd = a.down.bits;
    for (int l0 = 0; l0 < L; l0 += kBatchMax) {
        const int n = batch_size(L - l0);
        for (int i = 0; i < n; ++i) b.lay[i] = stack_desc(layers[l0 + i]);
        b.x = reinterpret_cast<const uint16_t*>(xb + l0 * step);
        b.y = reinterpret_cast<uint16_t*>(yb + l0 * step);
        unsigned* ctl = reinterpret_cast<unsigned*>(base);
        auto* t64 = reinterpret_cast<unsigned long long*>(b.t);
        hipError_t e = b.r == 0 || path == BatchPath::kStreamed ? hipSuccess   // streamed: in gate/up
                       : path == BatchPath::kMfma              ? launch_lora_a_mfma(b, n, st)
                                                               : launch_lora_a_batch(b, n, st);
        if (e == hipSuccess)
            e = path == BatchPath::kStreamed ? launch_gateup_stream(b, n, t64, ctl, st)
                : path == BatchPath::kMfma   ? launch_gateup_mfma(b, n, st)
                                             : launch_gateup_batch(b, n, st);
        if (e == hipSuccess)
            e = path == BatchPath::kStreamed ? launch_down_stream(b, n, ctl, st)
                : path == BatchPath::kMfma   ? launch_down_mfma(b, n, st)
                                             : launch_down_batch(b, n, st);
        if (e != hipSuccess)
            return QMLP_ERR_HIP;
    }
    return QMLP_OK;
}

}  // namespace

namespace qmlp {

// Everything qmlp_forward checks before it looks at the workspace.
qmlp_status forward_check(const qmlp_mlp* mlp, const void* x, int M, qmlp_dtype dtype, const void* y) {
    qmlp_status s = check_mlp(mlp, M, dtype);
    if (s != QMLP_OK)
        return s;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y))
        return QMLP_ERR_ALIGN;
    return QMLP_OK;
}

}  // namespace qmlp

extern "C" {

size_t qmlp_codes_bytes(int bits, int n_out, int k_in) {
    if (bits < 2 || bits > 4 || n_out <= 0 || k_in <= 0)
        return 0;
    // 3 bits: rows of 3k/8 bytes stay 16-byte aligned for k % 128 == 0
    if (bits == 3 ? k_in % 128 != 0 : k_in % (32 / bits) != 0)
        return 0;
    return (size_t)n_out * (size_t)k_in * (size_t)bits / 8;
}

size_t qmlp_meta_bytes(int n_out, int k_in, int group) {
    if (n_out <= 0 || k_in <= 0 || group <= 0 || k_in % group != 0)
        return 0;
    return (size_t)n_out * (size_t)(k_in / group) * 4;
}

size_t qmlp_workspace_bytes(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    if (check_mlp(mlp, M, dtype) != QMLP_OK)
        return 0;
    if (M == 0)
        return 0;
    return ws_total_bytes(mlp, M, dtype);
}

qmlp_status qmlp_pack_w2(const float* W, int n_out, int k_in, int group, qmlp_qweight* out,
                         int32_t* d_status, qmlp_stream stream) {
    return pack_common(2, W, n_out, k_in, group, out, d_status, stream);
}

qmlp_status qmlp_pack_w3(const float* W, int n_out, int k_in, int group, qmlp_qweight* out,
                         int32_t* d_status, qmlp_stream stream) {
    return pack_common(3, W, n_out, k_in, group, out, d_status, stream);
}

qmlp_status qmlp_pack_w4(const float* W, int n_out, int k_in, int group, qmlp_qweight* out,
                         int32_t* d_status, qmlp_stream stream) {
    return pack_common(4, W, n_out, k_in, group, out, d_status, stream);
}

qmlp_status qmlp_gateup_w2_lora(const qmlp_mlp* mlp, const void* x, int M, qmlp_dtype dtype,
                                void* h, void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = check_mlp(mlp, M, dtype);
    if (s != QMLP_OK)
        return s;
    if (mlp->gate.bits != 2)
        return QMLP_ERR_UNSUPPORTED;
    if (M == 0)
        return QMLP_OK;
    if (!x || !h)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(h))
        return QMLP_ERR_ALIGN;
    if (!ws || ws_bytes < qmlp_workspace_bytes(mlp, M, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    Workspace w = carve(mlp, M, dtype, ws);
    if (dtype == QMLP_BF16)
        return run_prefill_gateup(mlp, x, M, static_cast<uint16_t*>(h), w,
                                  static_cast<hipStream_t>(stream));
    return run_gateup(mlp, x, M, static_cast<uint16_t*>(h), w.t, static_cast<hipStream_t>(stream));
}

qmlp_status qmlp_down_w4(const qmlp_qweight* down, const void* h, int M, qmlp_dtype dtype,
                         void* y, qmlp_stream stream) {
    qmlp_status s = check_qweight(down, 4);
    if (s != QMLP_OK)
        return s;
    if (down->k_in % 64 != 0 || down->n_out % 64 != 0)
        return QMLP_ERR_SHAPE;
    if (M < 0)
        return QMLP_ERR_SHAPE;
    if (dtype == QMLP_BF16) {
        if (down->group == 32 || (M != 0 && (M % 128 != 0 || down->n_out % 128 != 0)))
            return QMLP_ERR_UNSUPPORTED;
    } else if (M > 16 || dtype != QMLP_F16 || !decode_shape_supported(down->n_out, down->k_in)) {
        return QMLP_ERR_UNSUPPORTED;
    }
    if (M == 0)
        return QMLP_OK;
    if (!h || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(h) || !aligned16(y))
        return QMLP_ERR_ALIGN;
    if (dtype == QMLP_BF16)
        return run_prefill_down(down, h, M, y, nullptr, static_cast<hipStream_t>(stream));
    return from_hip(launch_down(down_args(down, h, M, y), static_cast<hipStream_t>(stream)));
}

qmlp_status qmlp_forward(const qmlp_mlp* mlp, const void* x, int M, qmlp_dtype dtype, void* y,
                         void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = qmlp::forward_check(mlp, x, M, dtype, y);
    if (s != QMLP_OK || M == 0)
        return s;
    if (!ws || ws_bytes < qmlp_workspace_bytes(mlp, M, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    Workspace w = carve(mlp, M, dtype, ws);
    if (dtype == QMLP_BF16) {
        s = run_prefill_gateup(mlp, x, M, w.h, w, st);
        if (s != QMLP_OK)
            return s;
        return run_prefill_down(&mlp->down, w.h, M, y, w.part, st);
    }
    if (standard_mlp(mlp) &&
        fused_supported(M, mlp->gate.k_in, mlp->gate.n_out, mlp->gate.group, mlp->rank))
        return from_hip(launch_fused(gateup_args(mlp, x, M, w.h, w.t),
                                     down_args(&mlp->down, w.h, M, y),
                                     static_cast<const uint16_t*>(mlp->A_gate),
                                     static_cast<const uint16_t*>(mlp->A_up), w.t64, w.h32, w.ctl,
                                     st));
    s = run_gateup(mlp, x, M, w.h, w.t, st);
    if (s != QMLP_OK)
        return s;
    return from_hip(launch_down(down_args(&mlp->down, w.h, M, y), st));
}

qmlp_status qmlp_unpack(const qmlp_qweight* w, uint8_t* codes, uint16_t* scales, uint16_t* zeros,
                        qmlp_stream stream) {
    qmlp_status s = check_inspect(w);
    if (s != QMLP_OK)
        return s;
    if (!codes || !scales || !zeros)
        return QMLP_ERR_NULL;
    if (((uintptr_t)scales & 1u) || ((uintptr_t)zeros & 1u))
        return QMLP_ERR_ALIGN;
    return from_hip(launch_unpack(w->bits, static_cast<const uint32_t*>(w->codes),
                                  static_cast<const uint32_t*>(w->meta), w->n_out, w->k_in,
                                  w->group, codes, scales, zeros, static_cast<hipStream_t>(stream)));
}

qmlp_status qmlp_dequant(const qmlp_qweight* w, uint16_t* w_f16, qmlp_stream stream) {
    qmlp_status s = check_inspect(w);
    if (s != QMLP_OK)
        return s;
    if (!w_f16)
        return QMLP_ERR_NULL;
    if ((uintptr_t)w_f16 & 1u)
        return QMLP_ERR_ALIGN;
    return from_hip(launch_dequant(w->bits, static_cast<const uint32_t*>(w->codes),
                                   static_cast<const uint32_t*>(w->meta), w->n_out, w->k_in,
                                   w->group, w_f16, static_cast<hipStream_t>(stream)));
}

int qmlp_forward_launches(const qmlp_mlp* mlp, int M, qmlp_dtype dtype) {
    if (check_mlp(mlp, M, dtype) != QMLP_OK || M == 0)
        return 0;
    if (dtype == QMLP_BF16)
        return (mlp->rank > 0 ? 4 : 2) +
               (prefill_down_slices(M, mlp->gate.k_in, mlp->gate.n_out) > 1 ? 1 : 0);
    if (standard_mlp(mlp) &&
        fused_supported(M, mlp->gate.k_in, mlp->gate.n_out, mlp->gate.group, mlp->rank))
        return 1;
    return mlp->rank > 0 ? 3 : 2;
}

size_t qmlp_stack_workspace_bytes(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_stack(layers, L, M, dtype) != QMLP_OK || M == 0)
        return 0;
    size_t n = stack_layer_ws(layers, M, dtype) + 3 * round256((size_t)M * layers[0].gate.k_in * 2);
    if (stack_persistent(layers, M, dtype))
        n += stack_ws_bytes(layers[0].gate.k_in, layers[0].gate.n_out, layers[0].rank);
    return n;
}

size_t qmlp_stack_error_offset(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_stack(layers, L, M, dtype) != QMLP_OK || M == 0 || !stack_persistent(layers, M, dtype))
        return 0;
    return stack_layer_ws(layers, M, dtype) + 3 * round256((size_t)M * layers[0].gate.k_in * 2) +
           stack_error_word_offset();
}

int qmlp_stack_launches(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_stack(layers, L, M, dtype) != QMLP_OK || M == 0)
        return 0;
    if (stack_persistent(layers, M, dtype))
        return (L + stack_max_layers() - 1) / stack_max_layers();
    int n = 0;
    for (int i = 0; i < L; ++i) n += qmlp_forward_launches(&layers[i], M, dtype) + 2;
    return n - 1;
}

qmlp_status qmlp_forward_stack(const qmlp_mlp* layers, int L, const void* x, int M, qmlp_dtype dtype,
                               void* y, void* x_out, void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = check_stack(layers, L, M, dtype);
    if (s != QMLP_OK)
        return s;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y) || (x_out && !aligned16(x_out)))
        return QMLP_ERR_ALIGN;
    if (!ws || ws_bytes < qmlp_stack_workspace_bytes(layers, L, M, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    const int d = layers[0].gate.k_in;
    const size_t step = (size_t)M * d * 2;
    const size_t lws = stack_layer_ws(layers, M, dtype);
    char* pp[2] = {static_cast<char*>(ws) + lws, static_cast<char*>(ws) + lws + round256(step)};
    uint16_t* ub = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + lws + 2 * round256(step));
    char* area = static_cast<char*>(ws) + lws + 3 * round256(step);
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* yb = static_cast<char*>(y);
    if (stack_persistent(layers, M, dtype)) {
        StackLayerDesc desc[64];
        const int per = stack_max_layers();
        const uint16_t* xin = static_cast<const uint16_t*>(x);
        for (int l0 = 0, c = 0; l0 < L; l0 += per, ++c) {
            const int n = L - l0 < per ? L - l0 : per;
            for (int i = 0; i < n; ++i) desc[i] = stack_desc(layers[l0 + i]);
            // a later launch reads the residual stream the previous one left
            uint16_t* xl = l0 + n == L ? static_cast<uint16_t*>(x_out) : reinterpret_cast<uint16_t*>(pp[c & 1]);
            hipError_t e = launch_stack(desc, n, d, layers[0].gate.n_out, layers[0].gate.group, layers[0].rank,
                                        xin, reinterpret_cast<uint16_t*>(yb + l0 * step), xl, area, st);
            if (e != hipSuccess)
                return QMLP_ERR_HIP;
            xin = xl;
        }
        return QMLP_OK;
    }
    // per block: u_l = RMSNorm(x_l), y_l = MLP_l(u_l), then x_{l+1} = x_l + y_l
    const void* xin = x;
    for (int i = 0; i < L; ++i) {
        if (launch_rmsnorm(static_cast<const uint16_t*>(xin), ub, M, d, st) != hipSuccess)
            return QMLP_ERR_HIP;
        s = qmlp_forward(&layers[i], ub, M, dtype, yb + i * step, ws, lws, st);
        if (s != QMLP_OK)
            return s;
        void* next = i + 1 == L ? x_out : pp[i & 1];
        if (next) {
            hipError_t e = launch_residual(static_cast<const uint16_t*>(xin),
                                           reinterpret_cast<const uint16_t*>(yb + i * step),
                                           static_cast<uint16_t*>(next), M * d, dtype == QMLP_BF16, st);
            if (e != hipSuccess)
                return QMLP_ERR_HIP;
        }
        xin = next;
    }
    return QMLP_OK;
}

size_t qmlp_layers_workspace_bytes(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_layers(layers, L, M, dtype) != QMLP_OK || M == 0)
        return 0;
    if (dtype == QMLP_F16)              // streamed, matrix-core or batched
        return kCtlBytes +
               batch_t_bytes(layers, batch_size(L), M,
                             layers_mfma(layers, L, M, dtype) ? kLoraSlices : layers_streamed(layers, L, M, dtype) ? 2 : 1) +
               batch_h_bytes(layers, batch_size(L), M);
    return qmlp_workspace_bytes(&layers[0], M, dtype);
}

int qmlp_layers_path(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_layers(layers, L, M, dtype) != QMLP_OK || M == 0)
        return 0;
    if (layers_streamed(layers, L, M, dtype))
        return 1;
    if (layers_mfma(layers, L, M, dtype))
        return 4;
    if (layers_batched(layers, L, M, dtype))
        return 2;
    return 3;
}

int qmlp_layers_launches(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_layers(layers, L, M, dtype) != QMLP_OK || M == 0)
        return 0;
    if (dtype == QMLP_F16)              // three launches per batch (two streamed or without adapters)
        return (L + kBatchMax - 1) / kBatchMax *
               (layers[0].rank > 0 && !layers_streamed(layers, L, M, dtype) ? 3 : 2);
    int n = 0;
    for (int i = 0; i < L; ++i) n += qmlp_forward_launches(&layers[i], M, dtype);
    return n;
}

qmlp_status qmlp_forward_layers(const qmlp_mlp* layers, int L, const void* x, int M, qmlp_dtype dtype,
                                void* y, void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = check_layers(layers, L, M, dtype);
    if (s != QMLP_OK)
        return s;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y))
        return QMLP_ERR_ALIGN;
    if (!ws || ws_bytes < qmlp_layers_workspace_bytes(layers, L, M, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    const int d = layers[0].gate.k_in;
    const size_t step = (size_t)M * d * 2;
    const char* xb = static_cast<const char*>(x);
    char* yb = static_cast<char*>(y);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (dtype == QMLP_F16)
        return run_layers_batched(layers, L, xb, M, yb, ws, st, batch_path(layers, L, M, dtype));
    for (int i = 0; i < L; ++i) {
        s = qmlp_forward(&layers[i], xb + i * step, M, dtype, yb + i * step, ws, ws_bytes, stream);
        if (s != QMLP_OK)
            return s;
    }
    return QMLP_OK;
}

size_t qmlp_batch_workspace_bytes(const qmlp_mlp* layers, int L, int M, qmlp_dtype dtype) {
    if (check_layers(layers, L, M, dtype) != QMLP_OK || M == 0 || dtype != QMLP_F16)
        return 0;
    return kCtlBytes + batch_t_bytes(layers, batch_size(L), M) + batch_h_bytes(layers, batch_size(L), M);
}

qmlp_status qmlp_forward_batch(const qmlp_mlp* layers, int L, const void* x, int M, qmlp_dtype dtype,
                               void* y, void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = check_layers(layers, L, M, dtype);
    if (s != QMLP_OK)
        return s;
    if (dtype != QMLP_F16)
        return QMLP_ERR_UNSUPPORTED;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y))
        return QMLP_ERR_ALIGN;
    if (!ws || ws_bytes < qmlp_batch_workspace_bytes(layers, L, M, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    return run_layers_batched(layers, L, static_cast<const char*>(x), M, static_cast<char*>(y), ws,
                              static_cast<hipStream_t>(stream), BatchPath::kBatched);
}

qmlp_status qmlp_linear_batch(const qmlp_qweight* w, int L, const void* x, int M, qmlp_dtype dtype,
                              void* y, qmlp_stream stream) {
    if (!w)
        return QMLP_ERR_NULL;
    if (L <= 0 || L > kBatchMax || M < 0)
        return QMLP_ERR_SHAPE;
    for (int i = 0; i < L; ++i) {
        const qmlp_status s = check_qweight(&w[i], 0);
        if (s != QMLP_OK)
            return s;
        if (w[i].n_out != w[0].n_out || w[i].k_in != w[0].k_in || w[i].group != w[0].group ||
            w[i].bits != w[0].bits)
            return QMLP_ERR_SHAPE;
    }
    const int n = w[0].n_out, k = w[0].k_in, bits = w[0].bits;
    if (n % 64 != 0 || k % 64 != 0)
        return QMLP_ERR_SHAPE;
    if (dtype != QMLP_F16 || M > 16 || bits == 3 || (bits == 2 && w[0].group == 32) ||
        !units_fit(k, bits))
        return QMLP_ERR_UNSUPPORTED;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y))
        return QMLP_ERR_ALIGN;
    BatchArgs b{};
    for (int i = 0; i < L; ++i) {
        b.lay[i].cd = static_cast<const uint32_t*>(w[i].codes);
        b.lay[i].md = static_cast<const uint32_t*>(w[i].meta);
    }
    b.h = const_cast<uint16_t*>(static_cast<const uint16_t*>(x));
    b.y = static_cast<uint16_t*>(y);
    b.M = M;
    b.d = n;
    b.f = k;
    b.gd = w[0].group;
    b.bd = bits;
    return from_hip(launch_down_batch(b, L, static_cast<hipStream_t>(stream)));
}

size_t qmlp_moe_workspace_bytes(const qmlp_mlp* experts, int E, int M, int k, qmlp_dtype dtype) {
    if (E < 1 || E > kBatchMax || k < 1 || k > E || M < 1 || M > 16 || M * k > kBatchMax ||
        dtype != QMLP_F16 || check_layers(experts, E, 1, dtype) != QMLP_OK)
        return 0;
    const int n = M * k;
    // control block, t as tagged 64-bit words, h, the instances' outputs
    return kCtlBytes + batch_t_bytes(experts, n, 1, 2) + batch_h_bytes(experts, n, 1) +
           round256((size_t)n * experts[0].gate.k_in * 2);
}

qmlp_status qmlp_forward_moe(const qmlp_mlp* experts, int E, const void* x, int M,
                             qmlp_dtype dtype, const int32_t* topk_idx, const float* topk_w, int k,
                             void* y, void* ws, size_t ws_bytes, qmlp_stream stream) {
    qmlp_status s = check_layers(experts, E, 1, dtype);
    if (s != QMLP_OK)
        return s;
    if (E > kBatchMax || k < 1 || k > E || M < 0)
        return QMLP_ERR_SHAPE;
    if (dtype != QMLP_F16 || M > 16 || M * k > kBatchMax)
        return QMLP_ERR_UNSUPPORTED;
    if (M == 0)
        return QMLP_OK;
    if (!x || !y || !topk_idx || !topk_w)
        return QMLP_ERR_NULL;
    if (!aligned16(x) || !aligned16(y) || ((uintptr_t)topk_idx & 3u) || ((uintptr_t)topk_w & 3u))
        return QMLP_ERR_ALIGN;
    if (!ws || ws_bytes < qmlp_moe_workspace_bytes(experts, E, M, k, dtype))
        return QMLP_ERR_WORKSPACE;
    if (!aligned16(ws))
        return QMLP_ERR_ALIGN;
    const qmlp_mlp& a = experts[0];
    const int n = M * k, d = a.gate.k_in;
    char* base = static_cast<char*>(ws);
    BatchArgs b{};
    for (int i = 0; i < E; ++i) b.lay[i] = stack_desc(experts[i]);
    b.route = topk_idx;
    b.nexp = E;
    b.xdiv = k;                                   // instance l runs token l / k
    b.x = static_cast<const uint16_t*>(x);
    unsigned* ctl = reinterpret_cast<unsigned*>(base);
    auto* t64 = reinterpret_cast<unsigned long long*>(base + kCtlBytes);
    b.h = reinterpret_cast<uint16_t*>(base + kCtlBytes + batch_t_bytes(&a, n, 1, 2));
    b.y = reinterpret_cast<uint16_t*>(base + kCtlBytes + batch_t_bytes(&a, n, 1, 2) +
                                      batch_h_bytes(&a, n, 1));
    b.M = 1;
    b.d = d;
    b.f = a.gate.n_out;
    b.r = a.rank;
    b.gg = a.gate.group;
    b.bg = a.gate.bits;
    b.gd = a.down.group;
    b.bd = a.down.bits;
    hipStream_t st = static_cast<hipStream_t>(stream);
    // LoRA-A runs in the gate/up launch (one token per instance: always
    // here); t is handed over as tagged words
    if (!gateup_routed_fits(b, n))
        return QMLP_ERR_UNSUPPORTED;
    hipError_t e = launch_gateup_routed_batch(b, n, t64, ctl, st);
    if (down_combine_fits(b, n)) {
        // each workgroup computes all k instances of its rows and adds them
        if (e == hipSuccess)
            e = launch_down_combine(b, n, topk_w, static_cast<uint16_t*>(y), ctl, st);
        return from_hip(e);
    }
    if (e == hipSuccess)
        e = launch_down_batch(b, n, st);
    if (e == hipSuccess)
        e = launch_moe_combine(b.y, topk_w, M, k, d, static_cast<uint16_t*>(y), ctl, st);
    return from_hip(e);
}

const char* qmlp_status_string(qmlp_status s) {
    // a C caller may pass any int: read its bytes as an int, since loading a
    // value outside the enumerators' range as the enum type is undefined here
    int v = 0;
    std::memcpy(&v, &s, sizeof v);
    switch (v) {
    case QMLP_OK: return "ok";
    case QMLP_ERR_NULL: return "null pointer";
    case QMLP_ERR_SHAPE: return "invalid shape";
    case QMLP_ERR_ALIGN: return "misaligned pointer";
    case QMLP_ERR_UNSUPPORTED: return "unsupported combination";
    case QMLP_ERR_WORKSPACE: return "workspace missing or too small";
    case QMLP_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

}  // extern "C"
