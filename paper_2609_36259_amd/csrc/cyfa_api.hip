// Host side of the C ABI declared in include/cyfa.h: argument validation,
// workspace layout and kernel dispatch.  Every check runs before the first
// launch, so a rejected call enqueues nothing and writes nothing.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "cyfa.h"
#include "cyfa_bwd.h"
#include "cyfa_mixer.h"
#include "cyfa_internal.h"
#include "cyfa_rows.h"

namespace cyfa {
int valu_chunk_max();
bool mfma_supported(const FwdParams &p);
size_t mfma_workspace_bytes(const FwdParams &p, int segments);
int mfma_auto_segments(const FwdParams &p);
int mfma_default_chunk();
hipError_t launch_fwd_mfma(const FwdParams &p, int segments, void *ws, hipStream_t s,
                           hipEvent_t ev_start, hipEvent_t ev_stop, const MixIn *mix = nullptr);
}  // namespace cyfa

namespace {

thread_local char g_last_error[512] = "";
thread_local hipEvent_t g_ev_start = nullptr;
thread_local hipEvent_t g_ev_stop = nullptr;

hipError_t mark(hipEvent_t ev, hipStream_t s) {
    return ev ? hipEventRecord(ev, s) : hipSuccess;
}

cyfa_status fail(cyfa_status st, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

cyfa_status ok() {
    g_last_error[0] = '\0';
    return CYFA_OK;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

constexpr size_t kWsAlign = 256;
size_t round_up(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

bool head_dim_ok(int d) { return d == 64 || d == 128 || d == 256; }

struct FwdPlan {
    bool mfma;
    bool narrow;    // the 64-row matrix-core kernel (m <= 63)
    int chunk;
    int segments;
    size_t ws_bytes;
};

// layer: the layer forward (cyfa_forward_mixer), which runs the 128-row kernel
cyfa_status plan_forward(const cyfa_fwd_desc *d, FwdPlan *plan, bool layer = false) {
    if (!d) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc is NULL");
    if (d->B < 1 || d->H < 1 || d->T < 0)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "need B >= 1, H >= 1, T >= 0 (got B=%d T=%d H=%d)",
                    d->B, d->T, d->H);
    if ((double)d->B * d->T * d->H * (d->d_k > d->d_v ? d->d_k : d->d_v) > 4.0e12)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "problem too large");
    if (d->d_k <= 0 || d->d_v <= 0)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "head dims must be positive");
    if (!head_dim_ok(d->d_k) || !head_dim_ok(d->d_v))
        return fail(CYFA_ERR_UNSUPPORTED, "head dims must be 64, 128 or 256 (got d_k=%d d_v=%d)",
                    d->d_k, d->d_v);
    if (d->m < 3 || d->m > cyfa::kMaxActiveWide || (d->m % 2) == 0)
        return fail(d->m > cyfa::kMaxActiveWide && (d->m % 2) == 1 ? CYFA_ERR_UNSUPPORTED
                                                                   : CYFA_ERR_INVALID_ARGUMENT,
                    "m must be odd and in [3, 255] (got %d)", d->m);
    const bool wide = d->m > cyfa::kMaxActive;
    if (wide && (d->d_k > 128 || d->d_v > 128))
        return fail(CYFA_ERR_UNSUPPORTED, "m > 127 (256 storage rows) supports head dims 64 and 128");
    if (d->dtype != CYFA_F32 && d->dtype != CYFA_BF16)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad dtype %d", d->dtype);
    if (d->kernel < CYFA_KERNEL_AUTO || d->kernel > CYFA_KERNEL_MFMA)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad kernel selector %d", d->kernel);
    if (!std::isfinite(d->scale)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scale must be finite");
    if (d->segments < 0 || d->segments > 1024)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "segments must be in [0, 1024]");
    if (d->chunk < 0) return fail(CYFA_ERR_INVALID_ARGUMENT, "chunk must be >= 0");

    cyfa::FwdParams probe{};
    probe.B = d->B; probe.T = d->T; probe.H = d->H; probe.dk = d->d_k; probe.dv = d->d_v;
    probe.m = d->m; probe.dtype = d->dtype;
    probe.chunk = d->chunk ? d->chunk : cyfa::mfma_default_chunk();
    const bool mfma_ok = wide ? cyfa::mfma_wide_supported(probe) : cyfa::mfma_supported(probe);
    bool use_mfma;
    if (d->kernel == CYFA_KERNEL_MFMA) {
        if (!mfma_ok)
            return fail(CYFA_ERR_UNSUPPORTED,
                        "matrix-core kernel needs dtype=BF16, chunk 32 or 64, and d_k=d_v=128 (m up to 255) "
                        "or d_k=d_v=256 (m <= 127)");
        use_mfma = true;
    } else if (d->kernel == CYFA_KERNEL_VALU) {
        use_mfma = false;
    } else {
        use_mfma = mfma_ok;          // chunk 0, 32 or 64 with bf16 and d = 128 or 256
    }
    plan->mfma = use_mfma;
    plan->narrow = use_mfma && !wide && !layer && cyfa::mfma_narrow_supported(probe);
    size_t ws = round_up(cyfa::readout_bytes(d->H, d->m));
    if (plan->narrow) {
        // m <= 63 on 64 storage rows: chunk groups of a sequence, one workgroup each
        probe.chunk = cyfa::mfma_default_chunk();
        plan->chunk = probe.chunk;
        plan->segments = d->segments ? d->segments : cyfa::mfma_narrow_auto_groups(probe);
        const int nchunks = (d->T + probe.chunk - 1) / probe.chunk;
        if (plan->segments > nchunks && nchunks > 0) plan->segments = nchunks;
        if (plan->segments < 1) plan->segments = 1;
        ws = round_up(cyfa::mfma_narrow_workspace_bytes(probe, plan->segments));   // no fp32 readout matrix
    } else if (use_mfma && wide) {
        // chunk groups of a sequence, one workgroup each
        probe.chunk = cyfa::mfma_default_chunk();
        plan->chunk = probe.chunk;
        plan->segments = d->segments ? d->segments : cyfa::mfma_wide_auto_groups(probe);
        const int nchunks = (d->T + probe.chunk - 1) / probe.chunk;
        if (plan->segments > nchunks && nchunks > 0) plan->segments = nchunks;
        if (plan->segments < 1) plan->segments = 1;
        ws = round_up(cyfa::mfma_wide_workspace_bytes(probe, plan->segments));   // no fp32 readout matrix
    } else if (use_mfma) {
        probe.chunk = cyfa::mfma_default_chunk();    // a requested 64 runs as two 32-token chunks
        plan->chunk = probe.chunk;
        plan->segments = d->segments ? d->segments : cyfa::mfma_auto_segments(probe);
        const int nchunks = (d->T + probe.chunk - 1) / probe.chunk;
        if (plan->segments > nchunks && nchunks > 0) plan->segments = nchunks;
        if (plan->segments < 1) plan->segments = 1;
        ws += round_up(cyfa::mfma_workspace_bytes(probe, plan->segments));
    } else {
        const int c = d->chunk ? d->chunk : cyfa::valu_chunk_max();
        if (c != 8 && c != 16)
            return fail(CYFA_ERR_UNSUPPORTED, "vector-ALU kernel supports chunk 8 or 16 (got %d)", c);
        probe.chunk = c;
        if (d->segments > 1 && !cyfa::valu_groups_supported(probe))
            return fail(CYFA_ERR_UNSUPPORTED,
                        "vector-ALU kernel runs several segments only for d_k, d_v <= 128 and m <= 127");
        plan->chunk = c;
        plan->segments = d->segments ? d->segments : cyfa::valu_auto_groups(probe);
        ws += round_up(cyfa::valu_group_workspace_bytes(probe, plan->segments));
    }
    plan->ws_bytes = ws;
    return CYFA_OK;
}

struct BwdPlan {
    int groups;
    int mfma;       // matrix-core backward (32-token chunks) rather than the vector-ALU one
    int chunk;
    size_t ws_bytes;
};

cyfa_status plan_backward(const cyfa_fwd_desc *d, BwdPlan *plan) {
    if (!d) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc is NULL");
    if (d->B < 1 || d->H < 1 || d->T < 0)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "need B >= 1, H >= 1, T >= 0 (got B=%d T=%d H=%d)",
                    d->B, d->T, d->H);
    if ((double)d->B * d->T * d->H * (d->d_k > d->d_v ? d->d_k : d->d_v) > 4.0e12)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "problem too large");
    if (d->d_k <= 0 || d->d_v <= 0)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "head dims must be positive");
    const bool dims = ((d->d_k == 64 || d->d_k == 128) && (d->d_v == 64 || d->d_v == 128)) ||
                      (d->d_k == 256 && d->d_v == 256);
    if (!dims)
        return fail(CYFA_ERR_UNSUPPORTED,
                    "backward head dims must be 64 or 128 each, or both 256 (got d_k=%d d_v=%d)", d->d_k, d->d_v);
    if (d->m < 3 || d->m > cyfa::kMaxActive || (d->m % 2) == 0)
        return fail(d->m > cyfa::kMaxActive && (d->m % 2) == 1 ? CYFA_ERR_UNSUPPORTED
                                                               : CYFA_ERR_INVALID_ARGUMENT,
                    "backward: m must be odd and in [3, 127] (got %d)", d->m);
    if (d->dtype != CYFA_F32 && d->dtype != CYFA_BF16)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad dtype %d", d->dtype);
    if (d->kernel != CYFA_KERNEL_AUTO && d->kernel != CYFA_KERNEL_VALU && d->kernel != CYFA_KERNEL_MFMA)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad kernel %d", d->kernel);
    if (!std::isfinite(d->scale)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scale must be finite");
    const bool mfma_ok = d->dtype == CYFA_BF16 && d->d_k == 128 && d->d_v == 128;
    if (d->kernel == CYFA_KERNEL_MFMA && !mfma_ok)
        return fail(CYFA_ERR_UNSUPPORTED, "matrix-core backward: BF16 with d_k = d_v = 128");
    const bool mfma = d->kernel == CYFA_KERNEL_MFMA ||
                      (d->kernel == CYFA_KERNEL_AUTO && mfma_ok && d->chunk != cyfa::kBwdChunk);
    const int chunk = mfma ? cyfa::kBwdMfmaChunk : cyfa::kBwdChunk;
    if (d->chunk != 0 && d->chunk != chunk)
        return fail(CYFA_ERR_UNSUPPORTED, "backward chunk must be 0 or %d on the %s kernels (got %d)", chunk,
                    mfma ? "matrix-core" : "vector-ALU", d->chunk);
    if (d->segments < 0 || d->segments > 1024)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "segments must be in [0, 1024]");
    const int nc = (d->T + chunk - 1) / chunk;
    int g = d->segments ? d->segments
                        : (mfma ? cyfa::bwd_mfma_auto_groups(d->B, d->T, d->H) : cyfa::bwd_auto_groups(d->B, d->T, d->H));
    if (g > nc) g = nc;
    if (g < 1) g = 1;
    const int cpg = nc > 0 ? (nc + g - 1) / g : 1;
    plan->groups = nc > 0 ? (nc + cpg - 1) / cpg : 1;
    plan->mfma = mfma;
    plan->chunk = chunk;
    plan->ws_bytes = mfma ? cyfa::bwd_mfma_workspace_bytes(d->B, d->T, d->H, plan->groups)
                          : cyfa::bwd_workspace_bytes(d->B, d->T, d->H, d->d_k, d->d_v, plan->groups);
    return CYFA_OK;
}

cyfa_status check_dec(const cyfa_dec_desc *d) {
    if (!d) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc is NULL");
    if (d->N < 1 || d->H < 1) return fail(CYFA_ERR_INVALID_ARGUMENT, "need N >= 1 and H >= 1");
    if ((double)d->N * d->H > 2.0e9) return fail(CYFA_ERR_INVALID_ARGUMENT, "too many streams");
    if (d->d_k <= 0 || d->d_v <= 0) return fail(CYFA_ERR_INVALID_ARGUMENT, "head dims must be positive");
    if (!head_dim_ok(d->d_k) || !head_dim_ok(d->d_v))
        return fail(CYFA_ERR_UNSUPPORTED, "head dims must be 64, 128 or 256");
    if (d->m < 3 || d->m > cyfa::kMaxActiveWide || (d->m % 2) == 0)
        return fail(d->m > cyfa::kMaxActiveWide && (d->m % 2) == 1 ? CYFA_ERR_UNSUPPORTED
                                                                   : CYFA_ERR_INVALID_ARGUMENT,
                    "m must be odd and in [3, 255] (got %d)", d->m);
    if (d->m > cyfa::kMaxActive && (d->d_k > 128 || d->d_v > 128))
        return fail(CYFA_ERR_UNSUPPORTED, "m > 127 (256 storage rows) supports head dims 64 and 128");
    if (d->dtype != CYFA_F32 && d->dtype != CYFA_BF16)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad dtype %d", d->dtype);
    if (!std::isfinite(d->scale)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scale must be finite");
    return CYFA_OK;
}

}  // namespace

namespace {
cyfa_status check_mixer(const cyfa_mixer_desc *d) {
    if (!d) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc is NULL");
    if (d->B < 1 || d->H < 1 || d->T < 0)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "need B >= 1, H >= 1, T >= 0");
    if ((double)d->B * d->T * d->H * (d->d_k > d->d_v ? d->d_k : d->d_v) > 4.0e12)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "problem too large");
    if (!head_dim_ok(d->d_k) || !head_dim_ok(d->d_v))
        return fail(CYFA_ERR_UNSUPPORTED, "head dims must be 64, 128 or 256");
    if (d->conv_size < 1 || d->conv_size > cyfa::kMixMaxConv)
        return fail(CYFA_ERR_UNSUPPORTED, "conv_size must be in [1, %d]", cyfa::kMixMaxConv);
    if (d->conv_act != 0 && d->conv_act != 1) return fail(CYFA_ERR_INVALID_ARGUMENT, "conv_act must be 0 or 1");
    if (!(d->eps > 0.f) || !std::isfinite(d->eps)) return fail(CYFA_ERR_INVALID_ARGUMENT, "eps must be > 0");
    if (d->dtype != CYFA_F32 && d->dtype != CYFA_BF16)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "bad dtype %d", d->dtype);
    return CYFA_OK;
}

// workspace of the layer forward beyond the forward's: the prologue's q, k, v when the
// ShortConv runs in its own kernel
size_t mixer_qkv_bytes(const cyfa_fwd_desc *d, const cyfa_mixer_weights *mw) {
    if (mw->fuse_conv) return 0;
    return 3 * round_up((size_t)d->B * d->T * d->H * 128 * 2);
}

cyfa::MixParams mixer_params(const cyfa_mixer_desc *d) {
    cyfa::MixParams p{};
    p.B = d->B; p.T = d->T; p.H = d->H; p.dk = d->d_k; p.dv = d->d_v;
    p.K = d->conv_size; p.act = d->conv_act; p.eps = d->eps; p.dtype = d->dtype;
    return p;
}
}  // namespace

extern "C" {

cyfa_status cyfa_forward_workspace_size(const cyfa_fwd_desc *desc, size_t *bytes) {
    if (!bytes) return fail(CYFA_ERR_INVALID_ARGUMENT, "bytes is NULL");
    FwdPlan plan;
    cyfa_status st = plan_forward(desc, &plan);
    if (st != CYFA_OK) return st;
    *bytes = plan.ws_bytes;
    return ok();
}

cyfa_status cyfa_forward(const cyfa_fwd_desc *desc, const void *q, const void *k, const void *v,
                         const float *delta, const float *log_alpha, const float *beta,
                         const float *R, const float *K0, const float *V0, const double *clock0,
                         void *o, float *K_out, float *V_out, double *clock_out,
                         float *logits_out, void *workspace, size_t workspace_bytes,
                         void *stream) {
    return cyfa_forward_lens(desc, q, k, v, delta, log_alpha, beta, R, nullptr, K0, V0, clock0, o, K_out,
                             V_out, clock_out, logits_out, workspace, workspace_bytes, stream);
}

}  // extern "C"

namespace {
// cyfa_forward_lens (lens or nothing) and cyfa_forward_varlen (cu_seqlens)
// mix: the layer forward (cyfa_forward_mixer): q, k, v are the raw projections,
// the gates come from mix, and o receives the layer output.
cyfa_status forward_impl(const cyfa_fwd_desc *desc, const void *q, const void *k, const void *v,
                         const float *delta, const float *log_alpha, const float *beta, const float *R,
                         const int32_t *lens, const int32_t *cu, const float *K0, const float *V0,
                         const double *clock0, void *o, float *K_out, float *V_out, double *clock_out,
                         float *logits_out, void *workspace, size_t workspace_bytes, void *stream,
                         const cyfa::MixIn *mix = nullptr) {
    FwdPlan plan;
    cyfa_status st = plan_forward(desc, &plan, mix != nullptr);
    if (st != CYFA_OK) return st;
    const bool has_tokens = desc->T > 0;
    if (has_tokens && (!q || !k || !v || (!delta && !mix) || !o))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "q, k, v, delta and o are required");
    const void *vec[] = {q, k, v, o, K0, V0, K_out, V_out};
    const char *vec_names[] = {"q", "k", "v", "o", "K0", "V0", "K_out", "V_out"};
    for (int i = 0; i < 8; ++i)
        if (vec[i] && !aligned(vec[i], 16))
            return fail(CYFA_ERR_INVALID_ARGUMENT, "%s must be 16-byte aligned", vec_names[i]);
    const void *sc[] = {delta, log_alpha, beta, R, logits_out, lens, cu};
    for (const void *p : sc)
        if (p && !aligned(p, 4)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    if ((clock0 && !aligned(clock0, 8)) || (clock_out && !aligned(clock_out, 8)))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "clock arrays must be 8-byte aligned");
    if ((K_out && (K_out == (const float *)V0 || (const void *)K_out == q || (const void *)K_out == k)) ||
        (V_out && (V_out == (const float *)K0 || (const void *)V_out == v)) ||
        (K_out && K_out == V_out) || (o && (o == (void *)K_out || o == (void *)V_out)))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias other arguments");
    if (!workspace || workspace_bytes < plan.ws_bytes)
        return fail(CYFA_ERR_WORKSPACE, "workspace of %zu bytes required (got %zu)", plan.ws_bytes,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, kWsAlign))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");

    cyfa::FwdParams p{};
    p.B = desc->B; p.T = desc->T; p.H = desc->H; p.dk = desc->d_k; p.dv = desc->d_v;
    p.m = desc->m; p.chunk = plan.chunk; p.segments = plan.segments; p.scale = desc->scale;
    p.dtype = desc->dtype;
    p.q = q; p.k = k; p.v = v; p.delta = delta; p.log_alpha = log_alpha; p.beta = beta; p.R = R;
    p.K0 = K0; p.V0 = V0; p.clock0 = clock0; p.o = o; p.K_out = K_out; p.V_out = V_out;
    p.clock_out = clock_out; p.logits = logits_out; p.lens = lens; p.cu = cu;

    hipStream_t s = static_cast<hipStream_t>(stream);
    char *ws = static_cast<char *>(workspace);
    float *M = reinterpret_cast<float *>(ws);
    hipError_t e;
    if (plan.narrow) {
        // forms its own 64 x 64 bf16 readout matrix
        e = cyfa::launch_fwd_mfma_narrow(p, plan.segments, ws, s, g_ev_start, g_ev_stop);
    } else if (plan.mfma && p.m > cyfa::kMaxActive) {
        // forms its own bf16 readout matrix and its transpose
        e = cyfa::launch_fwd_mfma_wide(p, plan.segments, ws, s, g_ev_start, g_ev_stop);
    } else if (plan.mfma) {
        // forms its own bf16 readout matrix
        e = cyfa::launch_fwd_mfma(p, plan.segments, ws, s, g_ev_start, g_ev_stop, mix);
    } else {
        e = p.m > cyfa::kMaxActive ? cyfa::launch_readout_prep_wide(p.H, p.m, R, M, s)
                                   : cyfa::launch_readout_prep(p.H, p.m, R, M, nullptr, 1.f, s);
        if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "readout prep launch: %s", hipGetErrorString(e));
        e = mark(g_ev_start, s);
        if (e == hipSuccess)
            e = cyfa::launch_fwd_valu(p, M, plan.segments, ws + round_up(cyfa::readout_bytes(p.H, p.m)), s);
        if (e == hipSuccess) e = mark(g_ev_stop, s);
    }
    if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "forward launch: %s", hipGetErrorString(e));
    return ok();
}
}  // namespace

extern "C" {

cyfa_status cyfa_forward_lens(const cyfa_fwd_desc *desc, const void *q, const void *k, const void *v,
                              const float *delta, const float *log_alpha, const float *beta,
                              const float *R, const int32_t *lens, const float *K0, const float *V0,
                              const double *clock0, void *o, float *K_out, float *V_out,
                              double *clock_out, float *logits_out, void *workspace,
                              size_t workspace_bytes, void *stream) {
    return forward_impl(desc, q, k, v, delta, log_alpha, beta, R, lens, nullptr, K0, V0, clock0, o, K_out,
                        V_out, clock_out, logits_out, workspace, workspace_bytes, stream);
}

cyfa_status cyfa_forward_mixer_workspace_size(const cyfa_fwd_desc *desc, const cyfa_mixer_weights *mw,
                                              size_t *bytes) {
    if (!desc || !mw || !bytes) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc, mw and bytes are required");
    cyfa_fwd_desc d2 = *desc;
    d2.kernel = CYFA_KERNEL_MFMA;
    FwdPlan plan;
    cyfa_status st = plan_forward(&d2, &plan, true);
    if (st != CYFA_OK) return st;
    *bytes = plan.ws_bytes + mixer_qkv_bytes(desc, mw);
    return ok();
}

cyfa_status cyfa_forward_mixer(const cyfa_fwd_desc *desc, const cyfa_mixer_weights *mw, const void *q_in,
                               const void *k_in, const void *v_in, const float *R, const int32_t *lens,
                               const float *K0, const float *V0, const double *clock0, void *out,
                               float *K_out, float *V_out, double *clock_out, float *logits_out,
                               void *workspace, size_t workspace_bytes, void *stream) {
    if (!desc || !mw) return fail(CYFA_ERR_INVALID_ARGUMENT, "desc and mw are required");
    if (desc->dtype != CYFA_BF16 || desc->d_k != 128 || desc->d_v != 128 || desc->m > cyfa::kMaxActive ||
        desc->kernel == CYFA_KERNEL_VALU)
        return fail(CYFA_ERR_UNSUPPORTED,
                    "the layer forward runs on the matrix-core kernel: BF16, d_k = d_v = 128, m <= 127");
    if (mw->conv_size < 1 || mw->conv_size > cyfa::kMixMaxConv)
        return fail(CYFA_ERR_UNSUPPORTED, "conv_size must be in [1, %d]", cyfa::kMixMaxConv);
    if (mw->conv_act != 0 && mw->conv_act != 1) return fail(CYFA_ERR_INVALID_ARGUMENT, "conv_act must be 0 or 1");
    if (mw->fuse_conv != 0 && mw->fuse_conv != 1) return fail(CYFA_ERR_INVALID_ARGUMENT, "fuse_conv must be 0 or 1");
    if (!(mw->eps > 0.f) || !std::isfinite(mw->eps)) return fail(CYFA_ERR_INVALID_ARGUMENT, "eps must be > 0");
    if (desc->T > 0 && !mw->z_delta) return fail(CYFA_ERR_INVALID_ARGUMENT, "z_delta is required");
    if (mw->z_alpha && !mw->A) return fail(CYFA_ERR_INVALID_ARGUMENT, "A is required with z_alpha");
    const void *sc[] = {mw->conv_q, mw->conv_k, mw->conv_v, mw->norm_q, mw->norm_k, mw->z_delta, mw->b_delta,
                        mw->z_alpha, mw->b_alpha, mw->A, mw->z_beta, mw->norm_o};
    for (const void *ptr : sc)
        if (ptr && !aligned(ptr, 4)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    if (mw->gate && !aligned(mw->gate, 16)) return fail(CYFA_ERR_INVALID_ARGUMENT, "gate must be 16-byte aligned");
    {
        const void *ins[] = {q_in, k_in, v_in, mw->gate, mw->z_delta, mw->z_alpha, mw->z_beta, R, K0, V0, lens};
        for (const void *in : ins)
            if (out && in == out) return fail(CYFA_ERR_INVALID_ARGUMENT, "out must not alias an input");
    }
    cyfa_fwd_desc d2 = *desc;
    d2.kernel = CYFA_KERNEL_MFMA;
    FwdPlan plan;
    cyfa_status st = plan_forward(&d2, &plan, true);
    if (st != CYFA_OK) return st;
    const size_t need = plan.ws_bytes + mixer_qkv_bytes(desc, mw);
    if (!workspace || workspace_bytes < need)
        return fail(CYFA_ERR_WORKSPACE, "workspace of %zu bytes required (got %zu)", need,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, kWsAlign)) return fail(CYFA_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
    if (desc->T > 0 && (!q_in || !k_in || !v_in || !out))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "q_in, k_in, v_in and out are required");
    cyfa::MixIn mix{};
    mix.wq = mw->conv_q; mix.wk = mw->conv_k; mix.wv = mw->conv_v; mix.gq = mw->norm_q; mix.gk = mw->norm_k;
    mix.z_delta = mw->z_delta; mix.b_delta = mw->b_delta; mix.z_alpha = mw->z_alpha; mix.b_alpha = mw->b_alpha;
    mix.A = mw->A; mix.z_beta = mw->z_beta; mix.gate = mw->gate; mix.g_o = mw->norm_o;
    mix.K = mw->conv_size; mix.act = mw->conv_act; mix.eps = mw->eps; mix.fuse_conv = mw->fuse_conv;
    const void *q = q_in, *k = k_in, *v = v_in;
    if (!mw->fuse_conv && desc->T > 0) {
        // ShortConv and QK RMSNorm in the streaming kernel, into the workspace past the
        // forward's own part
        char *buf = static_cast<char *>(workspace) + plan.ws_bytes;
        const size_t one = mixer_qkv_bytes(desc, mw) / 3;
        cyfa::MixParams mp{};
        mp.B = desc->B; mp.T = desc->T; mp.H = desc->H; mp.dk = 128; mp.dv = 128;
        mp.K = mw->conv_size; mp.act = mw->conv_act; mp.eps = mw->eps; mp.dtype = CYFA_BF16;
        mp.q_in = q_in; mp.k_in = k_in; mp.v_in = v_in;
        mp.wq = mw->conv_q; mp.wk = mw->conv_k; mp.wv = mw->conv_v; mp.gq = mw->norm_q; mp.gk = mw->norm_k;
        mp.lens = lens;
        mp.q_out = buf; mp.k_out = buf + one; mp.v_out = buf + 2 * one;
        hipError_t e = cyfa::launch_mixer_prologue(mp, static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "mixer prologue launch: %s", hipGetErrorString(e));
        q = mp.q_out; k = mp.k_out; v = mp.v_out;
    }
    return forward_impl(&d2, q, k, v, nullptr, nullptr, nullptr, R, lens, nullptr, K0, V0, clock0, out,
                        K_out, V_out, clock_out, logits_out, workspace, plan.ws_bytes, stream, &mix);
}

cyfa_status cyfa_forward_varlen(const cyfa_fwd_desc *desc, const void *q, const void *k, const void *v,
                                const float *delta, const float *log_alpha, const float *beta,
                                const float *R, const int32_t *cu_seqlens, const float *K0, const float *V0,
                                const double *clock0, void *o, float *K_out, float *V_out,
                                double *clock_out, float *logits_out, void *workspace,
                                size_t workspace_bytes, void *stream) {
    if (!cu_seqlens) return fail(CYFA_ERR_INVALID_ARGUMENT, "cu_seqlens is required");
    return forward_impl(desc, q, k, v, delta, log_alpha, beta, R, nullptr, cu_seqlens, K0, V0, clock0, o, K_out,
                        V_out, clock_out, logits_out, workspace, workspace_bytes, stream);
}

cyfa_status cyfa_backward_workspace_size(const cyfa_fwd_desc *desc, size_t *bytes) {
    if (!bytes) return fail(CYFA_ERR_INVALID_ARGUMENT, "bytes is NULL");
    BwdPlan plan;
    cyfa_status st = plan_backward(desc, &plan);
    if (st != CYFA_OK) return st;
    *bytes = plan.ws_bytes;
    return ok();
}

cyfa_status cyfa_backward(const cyfa_fwd_desc *desc, const void *q, const void *k, const void *v,
                          const float *delta, const float *log_alpha, const float *beta,
                          const float *R, const int32_t *lens, const float *K0, const float *V0,
                          const double *clock0, const void *d_o, const float *dK_T,
                          const float *dV_T, void *dq, void *dk, void *dv, float *d_delta,
                          float *d_log_alpha, float *d_beta, float *d_R, float *d_K0, float *d_V0,
                          double *d_clock0, void *workspace, size_t workspace_bytes, void *stream) {
    BwdPlan plan;
    cyfa_status st = plan_backward(desc, &plan);
    if (st != CYFA_OK) return st;
    if (desc->T > 0 && (!q || !k || !v || !delta || !d_o || !dq || !dk || !dv || !d_delta))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "q, k, v, delta, d_o, dq, dk, dv and d_delta are required");
    if ((d_log_alpha && !log_alpha) || (d_beta && !beta) || (d_R && !R))
        return fail(CYFA_ERR_INVALID_ARGUMENT,
                    "the gradient of an input passed as NULL must be NULL (d_log_alpha, d_beta, d_R)");
    const void *vec[] = {q, k, v, d_o, K0, V0, dK_T, dV_T, dq, dk, dv, d_K0, d_V0};
    for (const void *p : vec)
        if (p && !aligned(p, 16)) return fail(CYFA_ERR_INVALID_ARGUMENT, "tensors must be 16-byte aligned");
    const void *sc[] = {delta, log_alpha, beta, R, lens, d_delta, d_log_alpha, d_beta, d_R};
    for (const void *p : sc)
        if (p && !aligned(p, 4)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    if ((clock0 && !aligned(clock0, 8)) || (d_clock0 && !aligned(d_clock0, 8)))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "clock arrays must be 8-byte aligned");
    {
        const void *outs[] = {dq, dk, dv, d_delta, d_log_alpha, d_beta, d_R, d_K0, d_V0, d_clock0};
        const void *ins[] = {q, k, v, delta, log_alpha, beta, R, lens, K0, V0, clock0, d_o, dK_T, dV_T};
        for (int a = 0; a < 10; ++a) {
            if (!outs[a]) continue;
            for (int c = a + 1; c < 10; ++c)
                if (outs[a] == outs[c]) return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias each other");
            for (const void *in : ins)
                if (in == outs[a]) return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias inputs");
        }
    }
    if (!workspace || workspace_bytes < plan.ws_bytes)
        return fail(CYFA_ERR_WORKSPACE, "workspace of %zu bytes required (got %zu)", plan.ws_bytes,
                    workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, kWsAlign))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");

    cyfa::BwdParams p{};
    p.B = desc->B; p.T = desc->T; p.H = desc->H; p.dk = desc->d_k; p.dv = desc->d_v; p.m = desc->m;
    p.nc = (desc->T + plan.chunk - 1) / plan.chunk;
    p.Tpad = p.nc * plan.chunk;
    p.groups = plan.groups;
    p.cpg = p.nc > 0 ? (p.nc + plan.groups - 1) / plan.groups : 1;
    p.scale = desc->scale; p.dtype = desc->dtype;
    p.q = q; p.k = k; p.v = v; p.dout = d_o;
    p.delta = delta; p.log_alpha = log_alpha; p.beta = beta; p.R = R; p.lens = lens;
    p.K0 = K0; p.V0 = V0; p.clock0 = clock0; p.dK_T = dK_T; p.dV_T = dV_T;
    p.gq = dq; p.gk = dk; p.gv = dv;
    p.gdelta = d_delta; p.glog_alpha = d_log_alpha; p.gbeta = d_beta; p.gR = d_R;
    p.gK0 = d_K0; p.gV0 = d_V0; p.gclock0 = d_clock0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = plan.mfma ? cyfa::launch_bwd_mfma(p, workspace, s) : cyfa::launch_bwd_valu(p, workspace, s);
    if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "backward launch: %s", hipGetErrorString(e));
    return ok();
}


cyfa_status cyfa_mixer_prologue(const cyfa_mixer_desc *desc, const void *q_in, const void *k_in,
                                const void *v_in, const float *conv_q, const float *conv_k,
                                const float *conv_v, const float *norm_q, const float *norm_k,
                                const float *z_delta, const float *b_delta, const float *z_alpha,
                                const float *b_alpha, const float *A, const float *z_beta,
                                const int32_t *lens, void *q, void *k, void *v, float *delta,
                                float *log_alpha, float *beta, void *stream) {
    cyfa_status st = check_mixer(desc);
    if (st != CYFA_OK) return st;
    if (desc->T > 0 && (!q_in || !k_in || !v_in || !q || !k || !v))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "q_in, k_in, v_in, q, k and v are required");
    if ((z_delta && !delta) || (z_alpha && (!log_alpha || !A)) || (z_beta && !beta))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "a gate projection needs its output (and A for z_alpha)");
    const void *vec[] = {q_in, k_in, v_in, q, k, v};
    for (const void *p : vec)
        if (p && !aligned(p, 16)) return fail(CYFA_ERR_INVALID_ARGUMENT, "tensors must be 16-byte aligned");
    const void *sc[] = {conv_q, conv_k, conv_v, norm_q, norm_k, z_delta, b_delta, z_alpha, b_alpha, A,
                        z_beta, lens, delta, log_alpha, beta};
    for (const void *p : sc)
        if (p && !aligned(p, 4)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    {
        const void *outs[] = {q, k, v, delta, log_alpha, beta};
        const void *ins[] = {q_in, k_in, v_in, conv_q, conv_k, conv_v, norm_q, norm_k, z_delta, b_delta,
                             z_alpha, b_alpha, A, z_beta, lens};
        for (int a = 0; a < 6; ++a) {
            if (!outs[a]) continue;
            for (int c = a + 1; c < 6; ++c)
                if (outs[a] == outs[c]) return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias each other");
            for (const void *in : ins)
                if (in == outs[a]) return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias inputs");
        }
    }
    cyfa::MixParams p = mixer_params(desc);
    p.q_in = q_in; p.k_in = k_in; p.v_in = v_in;
    p.wq = conv_q; p.wk = conv_k; p.wv = conv_v; p.gq = norm_q; p.gk = norm_k;
    p.z_delta = z_delta; p.b_delta = b_delta; p.z_alpha = z_alpha; p.b_alpha = b_alpha; p.A = A;
    p.z_beta = z_beta; p.lens = lens;
    p.q_out = q; p.k_out = k; p.v_out = v; p.delta = delta; p.log_alpha = log_alpha; p.beta = beta;
    hipError_t e = cyfa::launch_mixer_prologue(p, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "mixer prologue launch: %s", hipGetErrorString(e));
    return ok();
}

cyfa_status cyfa_mixer_epilogue(const cyfa_mixer_desc *desc, const void *o, const void *gate,
                                const float *norm_o, const int32_t *lens, void *out, void *stream) {
    cyfa_status st = check_mixer(desc);
    if (st != CYFA_OK) return st;
    if (desc->T > 0 && (!o || !out)) return fail(CYFA_ERR_INVALID_ARGUMENT, "o and out are required");
    const void *vec[] = {o, gate, out};
    for (const void *p : vec)
        if (p && !aligned(p, 16)) return fail(CYFA_ERR_INVALID_ARGUMENT, "tensors must be 16-byte aligned");
    if ((norm_o && !aligned(norm_o, 4)) || (lens && !aligned(lens, 4)))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    if (out && (out == o || out == gate)) return fail(CYFA_ERR_INVALID_ARGUMENT, "out must not alias o or gate");
    cyfa::MixParams p = mixer_params(desc);
    p.lens = lens;
    hipError_t e = cyfa::launch_mixer_epilogue(p, o, gate, norm_o, out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "mixer epilogue launch: %s", hipGetErrorString(e));
    return ok();
}

}  // extern "C"

// Scratch of cyfa_decode_step_noalloc: one copy per GPU, for the life of the
// process.  In host code `scratch` names a host-side stand-in, never the device
// memory: its device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[CYFA_DECODE_NOALLOC_SCRATCH_BYTES];

namespace {

cyfa_status check_decode_args(const cyfa_dec_desc *desc, const void *q, const void *k, const void *v,
                              const float *delta, const float *log_alpha, const float *beta,
                              const float *R, float *K, float *V, double *clock, void *o,
                              float *logits_out) {
    cyfa_status st = check_dec(desc);
    if (st != CYFA_OK) return st;
    if (!q || !k || !v || !delta || !K || !V || !clock || !o)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "q, k, v, delta, K, V, clock and o are required");
    const void *vec[] = {q, k, v, o, K, V};
    for (const void *p : vec)
        if (!aligned(p, 16)) return fail(CYFA_ERR_INVALID_ARGUMENT, "tensors must be 16-byte aligned");
    const void *sc[] = {delta, log_alpha, beta, R, logits_out};
    for (const void *p : sc)
        if (p && !aligned(p, 4)) return fail(CYFA_ERR_INVALID_ARGUMENT, "scalar arrays must be 4-byte aligned");
    if (!aligned(clock, 8)) return fail(CYFA_ERR_INVALID_ARGUMENT, "clock must be 8-byte aligned");
    if (K == V || o == (void *)K || o == (void *)V)
        return fail(CYFA_ERR_INVALID_ARGUMENT, "outputs must not alias each other");
    return CYFA_OK;
}

// Both decode entry points: readout matrices into M (every entry written), then
// the step.
cyfa_status run_decode(const cyfa_dec_desc *desc, const void *q, const void *k, const void *v,
                       const float *delta, const float *log_alpha, const float *beta, const float *R,
                       float *K, float *V, double *clock, void *o, float *logits_out, float *M,
                       hipStream_t s) {
    cyfa::DecParams p{};
    p.N = desc->N; p.H = desc->H; p.dk = desc->d_k; p.dv = desc->d_v; p.m = desc->m;
    p.scale = desc->scale; p.dtype = desc->dtype;
    p.q = q; p.k = k; p.v = v; p.delta = delta; p.log_alpha = log_alpha; p.beta = beta; p.R = R;
    p.K = K; p.V = V; p.clock = clock; p.o = o; p.logits = logits_out;
    hipError_t e = p.m > cyfa::kMaxActive ? cyfa::launch_readout_prep_wide(p.H, p.m, R, M, s)
                                          : cyfa::launch_readout_prep(p.H, p.m, R, M, nullptr, 1.f, s);
    if (e == hipSuccess) e = mark(g_ev_start, s);
    if (e == hipSuccess) e = cyfa::launch_decode(p, M, s);
    if (e == hipSuccess) e = mark(g_ev_stop, s);
    if (e != hipSuccess) return fail(CYFA_ERR_LAUNCH, "decode launch: %s", hipGetErrorString(e));
    return ok();
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (looked up on first use).
cyfa_status scratch_for_stream(hipStream_t s, float **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(CYFA_ERR_LAUNCH, "no usable current device");
    if (s) {
        int sdev = -1;
        if (hipStreamGetDevice(s, &sdev) != hipSuccess)
            return fail(CYFA_ERR_INVALID_ARGUMENT, "cannot query the stream's device");
        if (sdev != dev)
            return fail(CYFA_ERR_INVALID_ARGUMENT,
                        "stream belongs to device %d but device %d is current", sdev, dev);
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(CYFA_ERR_LAUNCH, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = static_cast<float *>(g_scratch_ptr[dev]);
    return CYFA_OK;
}

}  // namespace

extern "C" {

cyfa_status cyfa_decode_workspace_size(const cyfa_dec_desc *desc, size_t *bytes) {
    if (!bytes) return fail(CYFA_ERR_INVALID_ARGUMENT, "bytes is NULL");
    cyfa_status st = check_dec(desc);
    if (st != CYFA_OK) return st;
    *bytes = round_up(cyfa::readout_bytes(desc->H, desc->m));
    return ok();
}

cyfa_status cyfa_decode_step(const cyfa_dec_desc *desc, const void *q, const void *k, const void *v,
                             const float *delta, const float *log_alpha, const float *beta,
                             const float *R, float *K, float *V, double *clock, void *o,
                             float *logits_out, void *workspace, size_t workspace_bytes,
                             void *stream) {
    cyfa_status st = check_decode_args(desc, q, k, v, delta, log_alpha, beta, R, K, V, clock, o, logits_out);
    if (st != CYFA_OK) return st;
    const size_t need = round_up(cyfa::readout_bytes(desc->H, desc->m));
    if (!workspace || workspace_bytes < need)
        return fail(CYFA_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (!aligned(workspace, kWsAlign))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
    return run_decode(desc, q, k, v, delta, log_alpha, beta, R, K, V, clock, o, logits_out,
                      static_cast<float *>(workspace), static_cast<hipStream_t>(stream));
}

cyfa_status cyfa_decode_step_noalloc(const cyfa_dec_desc *desc, const void *q, const void *k, const void *v,
                                     const float *delta, const float *log_alpha, const float *beta,
                                     const float *R, float *K, float *V, double *clock, void *o,
                                     float *logits_out, void *stream) {
    cyfa_status st = check_decode_args(desc, q, k, v, delta, log_alpha, beta, R, K, V, clock, o, logits_out);
    if (st != CYFA_OK) return st;
    const size_t need = cyfa::readout_bytes(desc->H, desc->m);
    if (need > CYFA_DECODE_NOALLOC_SCRATCH_BYTES)
        return fail(CYFA_ERR_UNSUPPORTED,
                    "decode scratch of %zu bytes (H = %d, m = %d) exceeds the fixed %u-byte array of the "
                    "no-allocation entry point; use cyfa_decode_step with a workspace",
                    need, desc->H, desc->m, (unsigned)CYFA_DECODE_NOALLOC_SCRATCH_BYTES);
    hipStream_t s = static_cast<hipStream_t>(stream);
    float *M = nullptr;
    st = scratch_for_stream(s, &M);
    if (st != CYFA_OK) return st;
    return run_decode(desc, q, k, v, delta, log_alpha, beta, R, K, V, clock, o, logits_out, M, s);
}

const char *cyfa_status_string(cyfa_status status) {
    switch (status) {
        case CYFA_OK: return "ok";
        case CYFA_ERR_INVALID_ARGUMENT: return "invalid argument";
        case CYFA_ERR_UNSUPPORTED: return "unsupported configuration";
        case CYFA_ERR_WORKSPACE: return "workspace missing or too small";
        case CYFA_ERR_LAUNCH: return "kernel launch failed";
    }
    return "unknown status";
}

const char *cyfa_last_error(void) { return g_last_error; }

cyfa_status cyfa_set_timing_events(void *start_event, void *stop_event) {
    if ((start_event == nullptr) != (stop_event == nullptr))
        return fail(CYFA_ERR_INVALID_ARGUMENT, "set both timing events or neither");
    g_ev_start = static_cast<hipEvent_t>(start_event);
    g_ev_stop = static_cast<hipEvent_t>(stop_event);
    return ok();
}

int32_t cyfa_version(void) { return 100; }

}  // extern "C"
