// extern "C" entry points of libvmoe: argument validation, then launches.
#include <math.h>

#include <mutex>

#include "common.h"

namespace vmoe {

// Launchers (one per source file).
size_t route_workspace_bytes(const Dims& D);
size_t route_bwd_workspace_bytes(const Dims& D);
vmoe_status route_launch(const Dims& D, const void* x, const void* wr, const float* bias,
                         const float* noise, int flags, float* logits, float* probs,
                         int32_t* idx, int32_t* slot, float* gate, int32_t* order, int32_t* counts,
                         int32_t* row_base, void* ws, hipStream_t st);
vmoe_status dispatch_launch(const Dims& D, const void* x, const int32_t* idx, const int32_t* slot,
                            const int32_t* row_base, void* xe, hipStream_t st);
vmoe_status combine_fwd_launch(const Dims& D, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* y, hipStream_t st);
vmoe_status combine_bwd_launch(const Dims& D, const void* dy, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* dye, float* dgate, hipStream_t st);
vmoe_status dispatch_bwd_launch(const Dims& D, const void* dxe, const int32_t* idx,
                                const int32_t* slot, const int32_t* row_base, float* dx,
                                hipStream_t st);
vmoe_status ffn_fwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* b1, const void* w2, const void* b2, void* act,
                           void* act_grad, void* ye, int sched, const int32_t* row_token,
                           hipStream_t st);
vmoe_status ffn_bwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* w2, const void* act, const void* act_grad, const void* dye,
                           void* dh, void* dxe, float* dw1, float* db1, float* dw2, float* db2,
                           int sched, const int32_t* row_token, hipStream_t st);
vmoe_status row_token_launch(const Dims& D, const int32_t* idx, const int32_t* slot,
                             const int32_t* row_base, int32_t* row_token, hipStream_t st);
vmoe_status fcr_device_launch(int n, const int32_t* mn, const int32_t* sat, const double* coef,
                              int budget, int32_t* units, hipStream_t st);
vmoe_status route_bwd_launch(const Dims& D, const void* x, const void* wr, const float* probs,
                             const int32_t* idx, const int32_t* slot, const float* dgate,
                             const float* dz_add, float* dx, float* dwr, void* ws,
                             hipStream_t st);
vmoe_status dispatch_route_bwd_launch(const Dims& D, const void* dxe, const int32_t* row_base,
                                      const void* x, const void* wr, const float* probs,
                                      const int32_t* idx, const int32_t* slot,
                                      const float* dgate, const float* dz_add, float* dx,
                                      float* dwr, void* ws, hipStream_t st);
size_t balance_workspace_bytes(const Dims& D);
vmoe_status balance_launch(const Dims& D, const float* logits, const float* bias,
                           const float* noise, const float* probs, float sigma, float w_imp,
                           float w_load, float* losses, float* imp, float* load, float* dlogits,
                           void* ws, hipStream_t st);

vmoe_status make_dims(const vmoe_shape* s, Dims* out) {
    if (!s || !out) return VMOE_ERR_INVALID_ARG;
    if (s->n_tokens < 0 || s->n_groups < 1 || s->n_tokens % s->n_groups != 0)
        return VMOE_ERR_INVALID_ARG;
    if (s->n_experts < 1 || s->n_experts > kMaxExperts) return VMOE_ERR_INVALID_ARG;
    if (s->k < 1 || s->k > s->n_experts) return VMOE_ERR_INVALID_ARG;
    if (s->d_model < 8 || s->d_model % 8 != 0 || s->d_ff < 8 || s->d_ff % 8 != 0)
        return VMOE_ERR_INVALID_ARG;
    if (s->dtype != VMOE_F32 && s->dtype != VMOE_BF16) return VMOE_ERR_INVALID_ARG;
    if (s->capacity_rounding != 0 && s->capacity_rounding != 1) return VMOE_ERR_INVALID_ARG;
    if (s->capacity_override < 0 || s->reserved != 0) return VMOE_ERR_INVALID_ARG;
    if (!(s->capacity_factor > 0.0) || !isfinite(s->capacity_factor)) return VMOE_ERR_INVALID_ARG;
    Dims D;
    D.N = s->n_tokens;
    D.G = s->n_groups;
    D.Ng = s->n_tokens / s->n_groups;
    D.d = s->d_model;
    D.f = s->d_ff;
    D.E = s->n_experts;
    D.k = s->k;
    D.dtype = s->dtype;
    if (s->capacity_override > 0) {
        D.C = s->capacity_override;
    } else {
        const double c = static_cast<double>(s->k) * static_cast<double>(D.Ng) *
                         s->capacity_factor / static_cast<double>(D.E);
        const double r = s->capacity_rounding == 1 ? ceil(c) : floor(c + 0.5);
        if (!(r < 2147483647.0)) return VMOE_ERR_INVALID_ARG;
        D.C = r < 1.0 ? 1 : static_cast<int>(r);
    }
    // every buffer index must fit comfortably in 64 bits and rows in 31 bits
    if (static_cast<long long>(D.G) * D.C > 0x7FFFFFFFLL) return VMOE_ERR_INVALID_ARG;
    // 32-bit addressing limits of the kernels (a legal shape beyond them is
    // refused rather than computed wrongly):
    // - a buffer resource spans one expert's operand and reads zeros at byte
    //   offsets >= 2^31 (the tail-mask offset), so every per-expert operand
    //   ([G*C, d or f] activations, [f, d] weights) stays below 2^31 bytes;
    // - expert-buffer rows (E*G*C) and element indices into the expert buffers
    //   and the token-major tensors ([N, d], [N, E]) are 32-bit integers;
    // - the router backward addresses a chunk of 128 token rows of dx (f32)
    //   with 32-bit byte offsets, so d < 2^22.
    const long long lim = 0x7FFFFFFFLL;
    const long long elem = D.dtype == VMOE_BF16 ? 2 : 4;
    const long long rows = static_cast<long long>(D.G) * D.C;
    const long long wide = D.d > D.f ? D.d : D.f;
    const long long er = rows * D.E;
    if (rows * wide * elem > lim || static_cast<long long>(D.f) * D.d * elem > lim ||
        er > lim || er * wide > lim ||
        static_cast<long long>(D.N) * (wide > D.E ? wide : D.E) > lim ||
        128LL * D.d * 4 > lim)
        return VMOE_ERR_UNSUPPORTED;
    *out = D;
    return VMOE_OK;
}

}  // namespace vmoe

using vmoe::Dims;
using vmoe::aligned16;
using vmoe::as_stream;

// Routing scratch of vmoe_route_noalloc: one static array per GPU, which the
// runtime places when it loads the library's code on that GPU and holds until
// the process ends. Host code never passes `scratch` itself to a kernel (on
// the host it only names the symbol); its device address is looked up once
// per GPU with that GPU current and kept in scratch_ptr.
static __device__ __align__(256) unsigned char scratch[VMOE_ROUTE_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

// The current GPU's copy of `scratch`, or nullptr on a HIP error.
void* scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return nullptr;
        scratch_ptr[dev] = p;
    }
    return scratch_ptr[dev];
}
}  // namespace

#define VMOE_TRY(expr)                       \
    do {                                     \
        vmoe_status _s = (expr);             \
        if (_s != VMOE_OK) return _s;        \
    } while (0)

static vmoe_status need(bool ok) { return ok ? VMOE_OK : VMOE_ERR_INVALID_ARG; }

// A device buffer argument: required (non-NULL) and 16-byte aligned.
static bool dev(const void* p) { return p != nullptr && aligned16(p); }
// An optional device buffer: NULL or 16-byte aligned.
static bool opt(const void* p) { return p == nullptr || aligned16(p); }

extern "C" {

int32_t vmoe_abi_version(void) { return VMOE_ABI_VERSION; }

const char* vmoe_status_string(int32_t s) {
    switch (s) {
        case VMOE_OK: return "ok";
        case VMOE_ERR_INVALID_ARG: return "invalid argument";
        case VMOE_ERR_UNSUPPORTED: return "unsupported";
        case VMOE_ERR_WORKSPACE: return "workspace too small";
        case VMOE_ERR_HIP: return "HIP launch failed";
        default: return "unknown status";
    }
}

int32_t vmoe_capacity(const vmoe_shape* shape) {
    Dims D;
    return vmoe::make_dims(shape, &D) == VMOE_OK ? D.C : -1;
}

size_t vmoe_route_workspace_bytes(const vmoe_shape* shape) {
    Dims D;
    return vmoe::make_dims(shape, &D) == VMOE_OK ? vmoe::route_workspace_bytes(D) : 0;
}

size_t vmoe_route_bwd_workspace_bytes(const vmoe_shape* shape) {
    Dims D;
    return vmoe::make_dims(shape, &D) == VMOE_OK ? vmoe::route_bwd_workspace_bytes(D) : 0;
}

vmoe_status vmoe_route(const vmoe_shape* shape, const void* x, const void* w_router,
                       const float* logit_bias, const float* noise, int32_t flags, float* logits,
                       float* probs, int32_t* expert_idx, int32_t* slot, float* gate,
                       int32_t* order, int32_t* counts, int32_t* row_base, void* workspace,
                       size_t workspace_bytes, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need((flags & ~VMOE_ROUTE_LOGITS_IN) == 0));
    const bool logits_in = (flags & VMOE_ROUTE_LOGITS_IN) != 0;
    VMOE_TRY(need(logits_in || (dev(x) && dev(w_router))));
    VMOE_TRY(need(opt(logit_bias) && opt(noise)));
    VMOE_TRY(need(dev(logits) && dev(probs) && dev(expert_idx) && dev(slot) && dev(gate) &&
                  dev(order) && dev(counts) && dev(row_base)));
    const size_t need_ws = vmoe::route_workspace_bytes(D);
    if (workspace_bytes < need_ws || (need_ws > 0 && !dev(workspace))) return VMOE_ERR_WORKSPACE;
    return vmoe::route_launch(D, x, w_router, logit_bias, noise, flags, logits, probs, expert_idx,
                              slot, gate, order, counts, row_base, workspace, as_stream(stream));
}

vmoe_status vmoe_route_noalloc(const vmoe_shape* shape, const void* x, const void* w_router,
                               const float* logit_bias, const float* noise, int32_t flags,
                               float* logits, float* probs, int32_t* expert_idx, int32_t* slot,
                               float* gate, int32_t* order, int32_t* counts, int32_t* row_base,
                               void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need((flags & ~VMOE_ROUTE_LOGITS_IN) == 0));
    const bool logits_in = (flags & VMOE_ROUTE_LOGITS_IN) != 0;
    VMOE_TRY(need(logits_in || (dev(x) && dev(w_router))));
    VMOE_TRY(need(opt(logit_bias) && opt(noise)));
    VMOE_TRY(need(dev(logits) && dev(probs) && dev(expert_idx) && dev(slot) && dev(gate) &&
                  dev(order) && dev(counts) && dev(row_base)));
    // the routing kernels leave no state in the scratch between calls and
    // need none of it cleared: each pass writes what it later reads
    if (vmoe::route_workspace_bytes(D) > VMOE_ROUTE_NOALLOC_SCRATCH_BYTES)
        return VMOE_ERR_WORKSPACE;
    void* ws = scratch_on_current_device();
    if (ws == nullptr) return VMOE_ERR_HIP;
    return vmoe::route_launch(D, x, w_router, logit_bias, noise, flags, logits, probs, expert_idx,
                              slot, gate, order, counts, row_base, ws, as_stream(stream));
}

vmoe_status vmoe_dispatch(const vmoe_shape* shape, const void* x, const int32_t* expert_idx,
                          const int32_t* slot, const int32_t* row_base, void* xe, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(x) && dev(expert_idx) && dev(slot) && dev(row_base) && dev(xe)));
    return vmoe::dispatch_launch(D, x, expert_idx, slot, row_base, xe, as_stream(stream));
}

static vmoe_status ffn_fwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                           const void* w1, const void* b1, const void* w2, const void* b2,
                           void* act, void* act_grad, void* ye, int sched, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(xe) && dev(counts) && dev(w1) && dev(b1) && dev(w2) && dev(b2) &&
                  dev(act) && dev(act_grad) && dev(ye)));
    return vmoe::ffn_fwd_launch(D, xe, counts, w1, b1, w2, b2, act, act_grad, ye, sched,
                                nullptr, as_stream(stream));
}

static vmoe_status ffn_bwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                           const void* w1, const void* w2, const void* act, const void* act_grad,
                           const void* dye, void* dh, void* dxe, float* dw1, float* db1,
                           float* dw2, float* db2, int sched, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(xe) && dev(counts) && dev(w1) && dev(w2) && dev(act) && dev(act_grad) &&
                  dev(dye) && dev(dh) && dev(dxe) && dev(dw1) && dev(db1) && dev(dw2) &&
                  dev(db2)));
    return vmoe::ffn_bwd_launch(D, xe, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1,
                                dw2, db2, sched, nullptr, as_stream(stream));
}

vmoe_status vmoe_expert_ffn_fwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                                const void* w1, const void* b1, const void* w2, const void* b2,
                                void* act, void* act_grad, void* ye, void* stream) {
    return ffn_fwd(shape, xe, counts, w1, b1, w2, b2, act, act_grad, ye, 0, stream);
}

vmoe_status vmoe_expert_ffn_fwd_quota(const vmoe_shape* shape, const void* xe,
                                      const int32_t* counts, const void* w1, const void* b1,
                                      const void* w2, const void* b2, void* act, void* act_grad,
                                      void* ye, void* stream) {
    return ffn_fwd(shape, xe, counts, w1, b1, w2, b2, act, act_grad, ye, 1, stream);
}

vmoe_status vmoe_combine_fwd(const vmoe_shape* shape, const void* ye, const int32_t* expert_idx,
                             const int32_t* slot, const int32_t* row_base, const float* gate,
                             void* y, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(ye) && dev(expert_idx) && dev(slot) && dev(row_base) && dev(gate) &&
                  dev(y)));
    return vmoe::combine_fwd_launch(D, ye, expert_idx, slot, row_base, gate, y, as_stream(stream));
}

vmoe_status vmoe_combine_bwd(const vmoe_shape* shape, const void* dy, const void* ye,
                             const int32_t* expert_idx, const int32_t* slot,
                             const int32_t* row_base, const float* gate, void* dye, float* dgate,
                             void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(dy) && dev(ye) && dev(expert_idx) && dev(slot) && dev(row_base) &&
                  dev(gate) && dev(dye) && dev(dgate)));
    return vmoe::combine_bwd_launch(D, dy, ye, expert_idx, slot, row_base, gate, dye, dgate,
                                    as_stream(stream));
}

vmoe_status vmoe_expert_ffn_bwd(const vmoe_shape* shape, const void* xe, const int32_t* counts,
                                const void* w1, const void* w2, const void* act,
                                const void* act_grad, const void* dye, void* dh, void* dxe,
                                float* dw1, float* db1, float* dw2, float* db2, void* stream) {
    return ffn_bwd(shape, xe, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1, dw2, db2, 0,
                   stream);
}

vmoe_status vmoe_expert_ffn_bwd_quota(const vmoe_shape* shape, const void* xe,
                                      const int32_t* counts, const void* w1, const void* w2,
                                      const void* act, const void* act_grad, const void* dye,
                                      void* dh, void* dxe, float* dw1, float* db1, float* dw2,
                                      float* db2, void* stream) {
    return ffn_bwd(shape, xe, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1, dw2, db2, 1,
                   stream);
}

// Gathered (dispatch-fused) expert MLP: bf16 only, x addressable by one
// 32-bit buffer range, the weight gradient's token list within its LDS limit.
static vmoe_status gather_ok(const Dims& D, bool bwd) {
    if (D.dtype != VMOE_BF16) return VMOE_ERR_UNSUPPORTED;
    if (static_cast<long long>(D.N) * D.d * 2 > vmoe::kGatherMaxBytes) return VMOE_ERR_UNSUPPORTED;
    if (bwd && static_cast<long long>(D.G) * D.C > vmoe::kGatherRows) return VMOE_ERR_UNSUPPORTED;
    return VMOE_OK;
}

vmoe_status vmoe_dispatch_ffn_fwd(const vmoe_shape* shape, const void* x,
                                  const int32_t* expert_idx, const int32_t* slot,
                                  const int32_t* row_base, const int32_t* counts, const void* w1,
                                  const void* b1, const void* w2, const void* b2,
                                  int32_t* row_token, void* act, void* act_grad, void* ye,
                                  void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(x) && dev(expert_idx) && dev(slot) && dev(row_base) && dev(counts) &&
                  dev(w1) && dev(b1) && dev(w2) && dev(b2) && dev(row_token) && dev(act) &&
                  dev(act_grad) && dev(ye)));
    VMOE_TRY(gather_ok(D, false));
    VMOE_TRY(vmoe::row_token_launch(D, expert_idx, slot, row_base, row_token, as_stream(stream)));
    return vmoe::ffn_fwd_launch(D, x, counts, w1, b1, w2, b2, act, act_grad, ye, 0, row_token,
                                as_stream(stream));
}

vmoe_status vmoe_expert_ffn_bwd_gather(const vmoe_shape* shape, const void* x,
                                       const int32_t* row_token, const int32_t* counts,
                                       const void* w1, const void* w2, const void* act,
                                       const void* act_grad, const void* dye, void* dh, void* dxe,
                                       float* dw1, float* db1, float* dw2, float* db2,
                                       void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(x) && dev(row_token) && dev(counts) && dev(w1) && dev(w2) && dev(act) &&
                  dev(act_grad) && dev(dye) && dev(dh) && dev(dxe) && dev(dw1) && dev(db1) &&
                  dev(dw2) && dev(db2)));
    VMOE_TRY(gather_ok(D, true));
    return vmoe::ffn_bwd_launch(D, x, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1, dw2,
                                db2, 0, row_token, as_stream(stream));
}

vmoe_status vmoe_fill_clamp_refill_device(int32_t n, const int32_t* min_units,
                                          const int32_t* sat_units, const double* coef,
                                          int32_t budget, int32_t* alloc_units, void* stream) {
    if (n < 0 || n > vmoe::kMaxExperts || budget < 0) return VMOE_ERR_INVALID_ARG;
    if (n > 0 && !(dev(min_units) && dev(sat_units) && dev(coef) && dev(alloc_units)))
        return VMOE_ERR_INVALID_ARG;
    return vmoe::fcr_device_launch(n, min_units, sat_units, coef, budget, alloc_units,
                                   as_stream(stream));
}

vmoe_status vmoe_dispatch_bwd(const vmoe_shape* shape, const void* dxe,
                              const int32_t* expert_idx, const int32_t* slot,
                              const int32_t* row_base, float* dx, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(dxe) && dev(expert_idx) && dev(slot) && dev(row_base) && dev(dx)));
    return vmoe::dispatch_bwd_launch(D, dxe, expert_idx, slot, row_base, dx, as_stream(stream));
}

vmoe_status vmoe_route_bwd(const vmoe_shape* shape, const void* x, const void* w_router,
                           const float* probs, const int32_t* expert_idx, const int32_t* slot,
                           const float* dgate, float* dx, float* dw_router, void* workspace,
                           size_t workspace_bytes, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(x) && dev(w_router) && dev(probs) && dev(expert_idx) && dev(slot) &&
                  dev(dgate) && dev(dx) && opt(dw_router)));
    const size_t need_ws = vmoe::route_bwd_workspace_bytes(D);
    if (workspace_bytes < need_ws || (need_ws > 0 && !dev(workspace))) return VMOE_ERR_WORKSPACE;
    return vmoe::route_bwd_launch(D, x, w_router, probs, expert_idx, slot, dgate, nullptr, dx,
                                  dw_router, workspace, as_stream(stream));
}

vmoe_status vmoe_dispatch_route_bwd(const vmoe_shape* shape, const void* dxe,
                                    const int32_t* row_base, const void* x, const void* w_router,
                                    const float* probs, const int32_t* expert_idx,
                                    const int32_t* slot, const float* dgate, float* dx,
                                    float* dw_router, void* workspace, size_t workspace_bytes,
                                    void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(dxe) && dev(row_base) && dev(x) && dev(w_router) && dev(probs) &&
                  dev(expert_idx) && dev(slot) && dev(dgate) && dev(dx) && opt(dw_router)));
    const size_t need_ws = vmoe::route_bwd_workspace_bytes(D);
    if (workspace_bytes < need_ws || (need_ws > 0 && !dev(workspace))) return VMOE_ERR_WORKSPACE;
    return vmoe::dispatch_route_bwd_launch(D, dxe, row_base, x, w_router, probs, expert_idx, slot,
                                           dgate, nullptr, dx, dw_router, workspace,
                                           as_stream(stream));
}

vmoe_status vmoe_dispatch_route_bwd_dlogits(const vmoe_shape* shape, const void* dxe,
                                            const int32_t* row_base, const void* x,
                                            const void* w_router, const float* probs,
                                            const int32_t* expert_idx, const int32_t* slot,
                                            const float* dgate, const float* dlogits, float* dx,
                                            float* dw_router, void* workspace,
                                            size_t workspace_bytes, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(dxe) && dev(row_base) && dev(x) && dev(w_router) && dev(probs) &&
                  dev(expert_idx) && dev(slot) && dev(dgate) && dev(dlogits) && dev(dx) &&
                  opt(dw_router)));
    const size_t need_ws = vmoe::route_bwd_workspace_bytes(D);
    if (workspace_bytes < need_ws || (need_ws > 0 && !dev(workspace))) return VMOE_ERR_WORKSPACE;
    return vmoe::dispatch_route_bwd_launch(D, dxe, row_base, x, w_router, probs, expert_idx, slot,
                                           dgate, dlogits, dx, dw_router, workspace,
                                           as_stream(stream));
}

size_t vmoe_balance_loss_workspace_bytes(const vmoe_shape* shape) {
    Dims D;
    return vmoe::make_dims(shape, &D) == VMOE_OK ? vmoe::balance_workspace_bytes(D) : 0;
}

vmoe_status vmoe_balance_loss(const vmoe_shape* shape, const float* logits,
                              const float* logit_bias, const float* noise, const float* probs,
                              float noise_std, float w_importance, float w_load, float* losses,
                              float* importance, float* load, float* dlogits, void* workspace,
                              size_t workspace_bytes, void* stream) {
    Dims D;
    VMOE_TRY(vmoe::make_dims(shape, &D));
    VMOE_TRY(need(dev(logits) && dev(probs) && dev(losses) && dev(dlogits) && opt(logit_bias) &&
                  opt(noise) && opt(importance) && opt(load)));
    VMOE_TRY(need(noise_std > 0.0f && isfinite(noise_std) && isfinite(w_importance) &&
                  isfinite(w_load)));
    const size_t need_ws = vmoe::balance_workspace_bytes(D);
    if (workspace_bytes < need_ws || (need_ws > 0 && !dev(workspace))) return VMOE_ERR_WORKSPACE;
    return vmoe::balance_launch(D, logits, logit_bias, noise, probs, noise_std, w_importance,
                                w_load, losses, importance, load, dlogits, workspace,
                                as_stream(stream));
}

}  // extern "C"
