// One kernel per MLP layer for decode (M <= 4 tokens, binary16), gfx950.
//
// The whole block -- LoRA-A projection, fused 2-bit gate/up with LoRA-B and
// SiLU(G) * U, and the 4-bit down projection (Sec. 3.1 Eq. (1), Sec. 3.3,
// Sec. 4.2) -- runs as one launch, the fused gate-activation-down operator of
// Sec. 5.  Decode is bound by loading weights, and on MI355X a dependent
// kernel boundary costs about as much time as streaming one projection's
// weights, so the layer is not split into kernels:
//
//   * every wave issues the loads of ALL its packed weights at kernel start:
//     its gate/up rows and its down rows (the down weights do not depend on
//     h, so they stream in while gate/up computes);
//   * a few waves compute t = [A_g; A_u] x and publish it; every block reads
//     it once, for the LoRA-B epilogue;
//   * each block publishes its rows of h; every block reads all of h and
//     finishes its down rows.
//
// Hand-offs between compute units carry their own validity: each published
// value sits in one aligned word together with a 16-bit tag that changes
// with every call (h: binary16 | tag << 16; t: fp32 bits | tag << 32), is
// written with a device-coherent store and read with device-coherent loads
// until every word shows the current tag.  A single-copy-atomic word that
// shows the tag holds the value written with it, so the hand-off costs one
// trip through the memory system: no counter, no flag, no wait for the
// producer's stores to complete, and no cache write-back or invalidate
// (agent-scope fences on this GPU act on a whole L2).
//
// The tag is the call counter kept in the control block (word 0), plus one,
// modulo 65535, plus one: never 0, so a zeroed workspace holds no valid
// word.  The last block of every call advances the counter.  The grid is
// one block per compute unit, so every block is resident and every wait
// ends; each wait is also bounded (it sets an error bit and proceeds).
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

constexpr int FW = 8;                          // waves per block
constexpr unsigned kSpinLimit = 1u << 18;      // polls before a wait gives up
constexpr size_t kFusedLds = 144 * 1024;       // one block per CU: most of the 160 KB LDS
constexpr int kLoadWindow = 0;                 // weight loads a wave keeps in flight (0: no bound)

struct FusedArgs {
    GateUpArgs gu;
    DownArgs dn;
    const uint16_t* Ag;
    const uint16_t* Au;
    unsigned long long* t64;                   // [grid][256] tagged t: per block [4][2r]
    uint32_t* h32;                             // [4][f]  tagged h
    unsigned* ctl;
    int gu_items;                              // gate/up wave-items (8 rows each)
    int dn_items;                              // down wave-items (64/SD rows each)
    int nguw;                                  // waves per block that hold a gate/up item
    int lds_stage;                             // bytes of the x' / h' staging area
    int gu_meta_bytes;                         // per-wave LDS bytes for gate/up metadata
    int wmeta_bytes;                           // per-wave LDS metadata area
};

// Control words (uint32 indices into the workspace head, each on its own
// 128-byte line): call counter, blocks finished, sticky error bits.
constexpr int C_EPOCH = 0, C_DONE = 32, C_ERR = 160;

// Waves take one of two roles (the role is wave-uniform and branched on a
// scalar, so every wave runs exactly one path and meets the same barriers):
//   gate/up waves (wave < nguw): metadata, gate/up codes, LoRA-B, then down
//     items -- a straight-line load sequence, so each slot's wait covers
//     exactly the loads before it and the gate/up math overlaps the stream;
//   staging waves (the rest): their down items, and on a few of them the
//     LoRA-A rows, computed while the gate/up waves work; the last wave also
//     collects t into LDS.
// The activation is staged first: with XW > 0 by the staging waves alone
// (XW words per thread: activation loads, LoRA-A row loads, conversion, and
// only then their down loads), so it is not queued behind the gate/up
// waves' weight stream; with XW == 0 (more activation words than staging
// threads can take) every wave issues its activation words before its
// weight loads and converts them after.
// LDS: [x' | (C,X) | plain x  -- later h' | (C,X)][t, 1 KB][per-wave metadata].
template <int MT, int JG, int KM, int KA, int SD, int JD, int NDN, int XW>
__global__ void __launch_bounds__(FW * 64)
fused_layer_kernel(FusedArgs fa) {
    constexpr int SG = 8, RPWG = 8, RPWD = 64 / SD;
    extern __shared__ uint4 smem[];
    const GateUpArgs& a = fa.gu;
    const DownArgs& b = fa.dn;
    unsigned* ctl = fa.ctl;
    const unsigned epoch = __builtin_amdgcn_readfirstlane(
        __hip_atomic_load(&ctl[C_EPOCH], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    const uint32_t tag = epoch % 65535u + 1u;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int G = gridDim.x;
    const int Ug = a.d / 64, Ud = b.f / 32;     // the whole row is one LDS chunk
    const int nguw = fa.nguw;
    char* lds = reinterpret_cast<char*>(smem);
    uint4* xs = smem;
    float2* cxg = reinterpret_cast<float2*>(smem + MT * Ug * 8);
    uint4* xplain = smem + MT * Ug * 8 + (MT * Ug * 8 + 15) / 16;
    float* ts = reinterpret_cast<float*>(lds + fa.lds_stage);
    uint4* wmeta = reinterpret_cast<uint4*>(lds + fa.lds_stage + 1024 + wave * fa.wmeta_bytes);
    uint4* wmeta_dn = wmeta + fa.gu_meta_bytes / 16;
    const int dn_meta_chunks = RPWD * (b.f / b.g) / 4;

    // 1. Activation loads first.
    const int st_tid = tid - nguw * 64, st_threads = (FW - nguw) * 64;
    XWord xw[XW > 0 ? XW : MT];
    if constexpr (XW == 0) {
#pragma unroll
        for (int k = 0; k < MT; ++k)
            xw[k] = stage_x_load<MT>(a.x, a.M, a.d, 0, Ug, tid + k * FW * 64);
    }

    // 2. Weight loads by role.  With XW > 0 the staging waves first load and
    //    stage the activation (and the LoRA-A rows) and every other load is
    //    issued after that block barrier: the activation then reaches the
    //    compute unit in one unloaded round trip instead of queueing behind
    //    the whole weight stream, which starts one round trip later.
    FGuItem<MT, SG, JG, KM> gi;
    FDnItem<MT, SD, JD> di[NDN];
    LoraRow<KA> lr;
    const int gitem = blockIdx.x + wave * G;
    const int c = blockIdx.x + G * (FW - 1 - wave);          // LoRA-A row of a staging wave
    const bool lora_wave = wave >= nguw && a.r > 0 && c < 2 * a.r;
    if constexpr (XW > 0) {
        if (wave >= nguw) {
#pragma unroll
            for (int k = 0; k < XW; ++k)
                xw[k] = stage_x_load<MT>(a.x, a.M, a.d, 0, Ug, st_tid + k * st_threads);
            if (lora_wave)
                lora_a_load(lr, fa.Ag, fa.Au, a.d, a.r, c, lane);
#pragma unroll
            for (int k = 0; k < XW; ++k)
                stage_x_store<MT>(xs, cxg, Ug, Ug, a.M, st_tid + k * st_threads, xw[k], xplain);
        }
        __syncthreads();
    }
    if (wave < nguw) {
        const bool real = gitem < fa.gu_items;
        fgu_load<MT, SG, JG, KM, kLoadWindow>(gi, a, (real ? gitem : 0) * RPWG, lane);
        if (!real)
            gi.ok = false;                      // a dummy item: computed, never stored
    } else if constexpr (XW == 0) {
        if (lora_wave)
            lora_a_load(lr, fa.Ag, fa.Au, a.d, a.r, c, lane);
    }
    // Down items: the last wave loads its own after it has collected t (a
    // wave's loads return in issue order, so a poll queued behind a wave's
    // share of the weight stream would wait for all of it).
    auto load_down = [&]() {
#pragma unroll
        for (int k = 0; k < NDN; ++k) {
            const int item = blockIdx.x + ((FW - 1 - wave) + k * FW) * G;
            const bool act = item < fa.dn_items;
            fdn_load<MT, SD, JD, kLoadWindow>(di[k], b, (act ? item : 0) * RPWD, act, lane);
        }
    };
    if (wave != FW - 1)
        load_down();

    // 3. Activation into LDS (XW == 0: waits for the activation loads only).
    if constexpr (XW == 0) {
#pragma unroll
        for (int k = 0; k < MT; ++k)
            stage_x_store<MT>(xs, cxg, Ug, Ug, a.M, tid + k * FW * 64, xw[k], xplain);
        __syncthreads();
    }

    // 4. Gate/up dot products as the stream arrives; meanwhile LoRA-A.
    if (wave < nguw) {
        fgu_meta_to_lds(gi, a, wmeta, lane);
        fgu_accumulate(gi, xs, cxg, Ug, a.d, a.g, reinterpret_cast<const uint32_t*>(wmeta), lane);
    } else {
        if (lora_wave)
            lora_a_finish<MT, KA>(lr, xplain, a.M, a.d, a.r, c, fa.t64, tag, G, lane);
        if (wave == FW - 1 && a.r > 0) {
            bool fail = false;
            const unsigned long long* tb = fa.t64 + (long)blockIdx.x * 256;    // this block's copy
            for (int i = lane; i < a.M * 2 * a.r; i += 64) {
                unsigned long long v = 0;
                for (unsigned it = 0; it < kSpinLimit; ++it) {
                    v = __hip_atomic_load(tb + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if ((uint32_t)(v >> 32) == tag)
                        break;
                    __builtin_amdgcn_s_sleep(2);
                }
                fail |= (uint32_t)(v >> 32) != tag;
                ts[i] = __uint_as_float((uint32_t)v);
            }
            if (fail)
                atomicOr(&ctl[C_ERR], 1u);
        }
        if (wave == FW - 1)
            load_down();
    }
    __syncthreads();                            // t in LDS
    if (wave < nguw)
        fgu_finish(gi, a, ts, fa.h32, tag, lane);

    // 5. Unpack the down codes of the first kPre items while the other
    //    blocks finish gate/up (as many as fit in registers next to the h
    //    reads; the rest are unpacked just before their use).
    constexpr int kPre = MT > 1 ? 0 : NDN * JD * 16 <= 96 ? NDN : (JD * 16 <= 96 ? 1 : 0);
#pragma unroll
    for (int k = 0; k < kPre; ++k)
        fdn_extract(di[k]);

    // 6. Read all of h as it is published: each thread re-reads only the
    //    staging words that do not yet show this call's tag.
    const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
        fa.h32, 0, b.M * b.f * 4, 0x00020000);
    uint4 hw[4 * MT];
    uint32_t pending = (1u << (4 * MT)) - 1u;
    for (unsigned it = 0; pending != 0u && it < kSpinLimit; ++it) {
#pragma unroll
        for (int k = 0; k < 4 * MT; ++k) {
            if (pending & (1u << k)) {
                bool ok;
                const uint4 v = stage_h_load_tagged<MT>(hrs, b.f, b.M, Ud, tid + k * FW * 64, tag, ok);
                if (ok) {
                    hw[k] = v;
                    pending &= ~(1u << k);
                }
            }
        }
        if (pending != 0u)
            __builtin_amdgcn_s_sleep(2);
    }
    if (pending != 0u)
        atomicOr(&ctl[C_ERR], 2u);
    __syncthreads();                            // every wave is done with x'

    // 7. Down projection over the staged intermediate.
    {
#pragma unroll
        for (int k = 0; k < NDN; ++k)
            fdn_meta_to_lds(di[k], b, wmeta_dn + k * dn_meta_chunks, lane);
        uint4* hs = smem;
        float2* cx = reinterpret_cast<float2*>(smem + MT * Ud * 4);
#pragma unroll
        for (int k = 0; k < 4 * MT; ++k)
            stage_h_store<MT>(hs, cx, Ud, Ud, b.M, tid + k * FW * 64, hw[k]);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < NDN; ++k) {
            if (k >= kPre)
                fdn_extract(di[k]);
            fdn_accumulate(di[k], hs, cx, Ud, b.f, b.g,
                           reinterpret_cast<const uint32_t*>(wmeta_dn + k * dn_meta_chunks), lane);
        }
    }
#pragma unroll
    for (int k = 0; k < NDN; ++k)
        fdn_finish(di[k], b, lane);

    // 8. The last block to finish advances the call counter (every block
    //    read it at its start) and clears the finish count.
    if (tid == 0) {
        const unsigned old = __hip_atomic_fetch_add(&ctl[C_DONE], 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        if (old == (unsigned)G - 1) {
            __hip_atomic_store(&ctl[C_DONE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&ctl[C_EPOCH], epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// --------------------------------------------------------------- host side
namespace {

// Compute units of the current device (an immutable device property, cached).
int cu_count() {
    static int cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 0;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cache[dev] = n;
    }
    return cache[dev];
}

struct FusedPlan {
    int mt, jg, km, ka, sd, jd, ndn, nguw, xw, grid, gu_items, dn_items;
    int lds_stage, gu_meta_bytes, wmeta_bytes;
    size_t lds;
    bool ok;
};

FusedPlan plan_fused(int M, int d, int f, int g, int r) {
    FusedPlan p{};
    p.ok = false;
    p.mt = mtile_for(M);
    if (p.mt > 4)
        return p;
    const int Ug = d / 64, Ud = f / 32, ng = d / g, ngd = f / g;
    if (lanes_gateup(Ug) != 8)
        return p;
    p.sd = lanes_down(Ud);
    p.jg = (Ug + 7) / 8;
    p.jd = (Ud + p.sd - 1) / p.sd;
    if (p.jg > 8 || (p.sd != 8 && p.sd != 64) || p.jd > 8)
        return p;
    // metadata loads: gate+up chunks of 8 rows (16 B each) over 64 lanes;
    // down: one 16-byte chunk per lane
    p.km = (2 * 8 * ng / 4 + 63) / 64;
    const int rpwd = 64 / p.sd;
    if (p.km > 4 || (rpwd * ngd) % 4 != 0 || rpwd * ngd / 4 > 64)
        return p;
    p.grid = cu_count();
    if (p.grid <= 0)
        return p;
    p.gu_items = (f + 7) / 8;
    p.dn_items = (d + rpwd - 1) / rpwd;
    p.nguw = (p.gu_items + p.grid - 1) / p.grid;
    if (p.nguw >= FW)                          // at least one staging wave
        return p;
    if (2 * r > p.grid * (FW - p.nguw))         // LoRA-A rows on staging waves
        return p;
    p.ndn = (p.dn_items + FW * p.grid - 1) / (FW * p.grid);
    if (p.ndn > 2)
        return p;
    // activation words per staging thread (0: every wave stages)
    const int xwords = p.mt * Ug * 4, st_threads = (FW - p.nguw) * 64;
    p.xw = (xwords + st_threads - 1) / st_threads;
    if (p.xw > 2)
        p.xw = 0;
    // The h' staging holds at most 4*MT words per thread.
    if (p.mt * Ud * 4 > 4 * p.mt * FW * 64 || Ug > 128)
        return p;
    p.ka = (d / 8 + 63) / 64;                   // LoRA-A chunks per lane (<= 8 as d <= 4096)
    // x' + (C, X) + the plain activation, or h' + (C, X)
    const size_t lg = (size_t)p.mt * Ug * GU_UNIT_BYTES + 16 + (size_t)p.mt * d * 2;
    const size_t ld = (size_t)p.mt * Ud * DN_UNIT_BYTES;
    p.lds_stage = (int)((lg > ld ? lg : ld) + 15) / 16 * 16;
    p.gu_meta_bytes = 2 * 8 * ng * 4;
    p.wmeta_bytes = p.gu_meta_bytes + p.ndn * rpwd * ngd * 4;
    p.lds = (size_t)p.lds_stage + 1024 + (size_t)FW * p.wmeta_bytes;
    // The generic 8-slot instance at 2 or 4 tokens with two down items a
    // wave does not fit in registers: such shapes take the three-kernel path.
    const bool exact = (p.jg == 5 && p.km == 2 && p.ka == 5 && p.sd == 64 && p.jd == 5 && p.ndn == 2) ||
                       (p.jg == 8 && p.km == 2 && p.ka == 8 && p.sd == 64 && p.jd == 6 && p.ndn == 2) ||
                       (p.jg == 1 && p.km == 1 && p.ka == 1 && p.sd == 8 && p.jd == 6 && p.ndn == 1);
    if (!exact)
        p.xw = 0;                               // generic instances stage with every wave
    if (!exact && p.mt >= 2 && p.ndn == 2)
        return p;
    p.ok = p.lds <= kFusedLds;
    return p;
}

}  // namespace

bool fused_supported(int M, int d, int f, int g, int r) { return plan_fused(M, d, f, g, r).ok; }

int fused_grid() { return cu_count(); }

// Exact slot counts for the common shapes, else the 8-slot generic instance
// (slots past the row are dummies).
#define QMLP_FU_EXACT(MT_, JG_, KM_, KA_, SD_, JD_, NDN_, XW_)                            \
    if (p.mt == MT_ && p.jg == JG_ && p.km == KM_ && p.ka == KA_ && p.sd == SD_ &&        \
        p.jd == JD_ && p.ndn == NDN_ && p.xw == XW_)                                      \
        return run(fused_layer_kernel<MT_, JG_, KM_, KA_, SD_, JD_, NDN_, XW_>);
#define QMLP_FU_GENERIC(MT_, SD_, NDN_)                                                   \
    if (p.mt == MT_ && p.sd == SD_ && p.ndn == NDN_)                                      \
        return run(fused_layer_kernel<MT_, 8, 4, 8, SD_, 8, NDN_, 0>);
#define QMLP_FU_MT(MT_)                                                                   \
    QMLP_FU_EXACT(MT_, 5, 2, 5, 64, 5, 2, 1) QMLP_FU_EXACT(MT_, 5, 2, 5, 64, 5, 2, 2)   \
    QMLP_FU_EXACT(MT_, 5, 2, 5, 64, 5, 2, 0)                                              \
    QMLP_FU_EXACT(MT_, 8, 2, 8, 64, 6, 2, 1) QMLP_FU_EXACT(MT_, 8, 2, 8, 64, 6, 2, 2)   \
    QMLP_FU_EXACT(MT_, 8, 2, 8, 64, 6, 2, 0)                                              \
    QMLP_FU_EXACT(MT_, 1, 1, 1, 8, 6, 1, 1) QMLP_FU_EXACT(MT_, 1, 1, 1, 8, 6, 1, 0)     \
    QMLP_FU_GENERIC(MT_, 8, 1) QMLP_FU_GENERIC(MT_, 64, 1)
#define QMLP_FU_MT2(MT_) QMLP_FU_GENERIC(MT_, 8, 2) QMLP_FU_GENERIC(MT_, 64, 2)

hipError_t launch_fused(GateUpArgs gu, DownArgs dn, const uint16_t* Ag, const uint16_t* Au,
                        unsigned long long* t64, uint32_t* h32, unsigned* ctl, hipStream_t st) {
    const FusedPlan p = plan_fused(gu.M, gu.d, gu.f, gu.g, gu.r);
    if (!p.ok)
        return hipErrorInvalidValue;
    gu.uc = gu.d / 64;
    dn.uc = dn.f / 32;
    FusedArgs fa{gu, dn, Ag, Au, t64, h32, ctl, p.gu_items, p.dn_items, p.nguw,
                 p.lds_stage, p.gu_meta_bytes, p.wmeta_bytes};
    auto run = [&](auto kernel) -> hipError_t {
        hipError_t e = set_lds(kernel, p.lds);
        if (e != hipSuccess)
            return e;
        kernel<<<p.grid, FW * 64, p.lds, st>>>(fa);
        return hipGetLastError();
    };
    QMLP_FU_MT(1) QMLP_FU_MT(2) QMLP_FU_MT(4) QMLP_FU_MT2(1)
    return hipErrorInvalidValue;
}

}  // namespace qmlp
