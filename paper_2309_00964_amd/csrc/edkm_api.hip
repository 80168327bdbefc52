// C ABI of the eDKM hot path: argument checks, per-plan call order, workspace
// layout, and the split of each batch into launches.  Every check runs on the
// host before any HIP call; kernels never see an argument this layer rejected.

#include "../../include/edkm.h"
#include "edkm_internal.h"
#include "edkm_partition.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>

namespace edkm {

namespace {

constexpr uint64_t PLAN_MAGIC = 0x65444B4D706C616EULL;   // "eDKMplan"
enum Stage : int32_t { PLANNED = 1, COUNTED = 2, FORWARD = 3, DENSE_FORWARD = 4 };

struct PlanImpl {
    uint64_t magic;
    const void* self;        // the record's own address: a copied record is refused
    uint64_t n;
    int32_t bits, k, max_iter, stage;
    int32_t fmt;             // FMT_FP16 or FMT_BF16
    int32_t kforce;          // EDKM_KEYED_AUTO, _I32 or _U64
    void* ws;
    size_t ws_bytes;
    const uint16_t* keys;   // key buffer of the current sequence
    float tau;
    float eps;
    int32_t hip_code;        // last HIP failure on this plan (0 if none)
    const char* hip_step;    // the launch or runtime call that failed
    PassEvents ev;           // caller's timing events (diagnostics), null when unset
};
static_assert(sizeof(PlanImpl) <= sizeof(edkm_plan), "edkm_plan too small");
static_assert(EDKM_KEYS_FP16 != EDKM_KEYS_BF16, "key formats");
static_assert(EDKM_NOALLOC_SCRATCH_BYTES == NOALLOC_SCRATCH_BYTES,
              "the header states the allocation-free palettization's device array size");
static_assert(EDKM_KEYED_I32 == KEYED_I32 && EDKM_KEYED_U64 == KEYED_U64, "keyed-sum modes");
static_assert(EDKM_PASS_HIST == PASS_HIST && EDKM_PASS_GATHER_WT == PASS_GATHER_WT &&
                  EDKM_PASS_KEYED_GRAD == PASS_KEYED_GRAD && EDKM_PASS_GATHER_GRAD == PASS_GATHER_GRAD &&
                  EDKM_PASS_DENSE_ITER == PASS_DENSE_ITER && EDKM_PASS_DENSE_BITER == PASS_DENSE_BITER &&
                  EDKM_PASS_PALETTIZE == PASS_PALETTIZE && EDKM_PASS_INVERSE == PASS_INVERSE,
              "pass ids");

inline PlanImpl* impl(edkm_plan* p) { return reinterpret_cast<PlanImpl*>(p); }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool plan_ok(const edkm_plan* p) {
    return p && reinterpret_cast<const PlanImpl*>(p)->magic == PLAN_MAGIC &&
           reinterpret_cast<const PlanImpl*>(p)->self == p;
}

// Workgroups one N-sized pass may use: one per compute unit of the current
// device (each workgroup holds a whole CU's LDS, so a larger grid would run a
// second, nearly empty wave), at most NP_MAX_WG.  Cached per device.
int np_budget() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return NP_MAX_WG;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus < 1)
            cus = NP_MAX_WG;
        v = std::min(cus, NP_MAX_WG);
        cache[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

// Split the N-sized passes of a group over at most `budget` workgroups
// (split_passes); the slices go into the matrices' launch arguments.
uint32_t partition(BatchArgs& b, int budget) {
    uint64_t n[MAXB], chunk[MAXB];
    uint32_t cnt[MAXB], beg[MAXB];
    for (int i = 0; i < b.count; ++i) n[i] = b.m[i].n;
    const uint32_t grid = split_passes(n, b.count, budget, NP_MIN_CHUNK, chunk, cnt, beg);
    for (int i = 0; i < b.count; ++i) {
        b.m[i].chunk = chunk[i];
        b.m[i].wg_count = cnt[i];
        b.wg_begin[i] = beg[i];
    }
    for (int i = b.count; i < MAXB; ++i) b.wg_begin[i] = 0xFFFFFFFFu;   // no workgroup reaches these
    return grid;
}

float tau_s2(float tau) { return (float)(1.4426950408889634 / (double)tau); }

// Record a HIP failure on plans[first .. first+cnt) and return EDKM_ERR_HIP.
edkm_status hip_fail(edkm_plan* const* plans, int first, int cnt, hipError_t e, const char* step) {
    for (int i = 0; i < cnt; ++i) {
        reinterpret_cast<PlanImpl*>(plans[first + i])->hip_code = (int32_t)e;
        reinterpret_cast<PlanImpl*>(plans[first + i])->hip_step = step;
    }
    return EDKM_ERR_HIP;
}

}  // namespace

namespace {

void fill_mat(MatArgs& M, const PlanImpl* P, const uint16_t* keys) {
    std::memset(&M, 0, sizeof(M));
    M.keys = keys;
    M.n = P->n;
    M.k = P->k;
    M.max_iter = P->max_iter;
    M.fmt = P->fmt;
    M.kforce = P->kforce;
    M.wsb = P->ws;
}

// Common checks of a batch: plans valid and distinct, key buffers non-null.
edkm_status check_batch(int count, edkm_plan* const* plans, const uint16_t* const* keys) {
    if (count < 1 || !plans || !keys) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i) {
        if (!plan_ok(plans[i]) || !keys[i]) return EDKM_ERR_ARG;
        for (int j = 0; j < i; ++j)
            if (plans[j] == plans[i] || impl(plans[j])->ws == impl(plans[i])->ws) return EDKM_ERR_ARG;
    }
    return EDKM_OK;
}

bool tau_ok(float tau) { return std::isfinite(tau) && tau > 0.f && std::isfinite(1.0f / tau); }
bool eps_ok(float eps) { return std::isfinite(eps) && eps >= 0.f; }

// Launch groups: consecutive matrices with the same k and weight format, at
// most MAXB each.
template <class Fn>
edkm_status for_groups(int count, edkm_plan* const* plans, Fn fn) {
    int i = 0;
    while (i < count) {
        int j = i + 1;
        while (j < count && j - i < MAXB && impl(plans[j])->k == impl(plans[i])->k &&
               impl(plans[j])->fmt == impl(plans[i])->fmt)
            ++j;
        edkm_status st = fn(i, j - i);
        if (st != EDKM_OK) return st;
        i = j;
    }
    return EDKM_OK;
}

}  // namespace
}  // namespace edkm

using namespace edkm;

extern "C" {

size_t edkm_workspace_bytes(uint64_t n, int bits, int max_iter) {
    if (n < 1 || n > EDKM_MAX_N || bits < 1 || bits > EDKM_MAX_BITS || max_iter < 1 ||
        max_iter > EDKM_MAX_ITER)
        return 0;
    return workspace_bytes(max_iter);
}

edkm_status edkm_plan_init(edkm_plan* plan, uint64_t n, int bits, int max_iter, void* ws,
                           size_t ws_bytes) {
    return edkm_plan_init_ex(plan, n, bits, max_iter, EDKM_KEYS_FP16, ws, ws_bytes);
}

edkm_status edkm_plan_init_ex(edkm_plan* plan, uint64_t n, int bits, int max_iter, int key_format,
                              void* ws, size_t ws_bytes) {
    if (!plan || (key_format != EDKM_KEYS_FP16 && key_format != EDKM_KEYS_BF16)) return EDKM_ERR_ARG;
    const size_t need = edkm_workspace_bytes(n, bits, max_iter);
    if (need == 0) return EDKM_ERR_ARG;
    if (!ws || ws_bytes < need || ((uintptr_t)ws & 255u)) return EDKM_ERR_WORKSPACE;
    std::memset(plan, 0, sizeof(*plan));
    PlanImpl* P = impl(plan);
    P->n = n;
    P->bits = bits;
    P->k = 1 << bits;
    P->max_iter = max_iter;
    P->fmt = key_format == EDKM_KEYS_BF16 ? FMT_BF16 : FMT_FP16;
    P->kforce = EDKM_KEYED_AUTO;
    P->ws = ws;
    P->ws_bytes = ws_bytes;
    P->stage = PLANNED;
    P->self = plan;
    P->magic = PLAN_MAGIC;
    return EDKM_OK;
}

edkm_status edkm_init_unique_batch(int count, edkm_plan* const* plans,
                                   const uint16_t* const* w_bits, uint32_t* const* counts_out,
                                   uint32_t* const* num_unique_out, int check_finite,
                                   hipStream_t stream) {
    edkm_status st = check_batch(count, plans, w_bits);
    if (st != EDKM_OK) return st;
    if (check_finite != 0 && check_finite != 1) return EDKM_ERR_ARG;
    // From the first launch on, the workspaces hold a partial count of the new
    // keys: until this call succeeds, every plan of it needs a new init_unique.
    for (int i = 0; i < count; ++i) {
        impl(plans[i])->stage = PLANNED;
        impl(plans[i])->keys = nullptr;
    }
    st = for_groups(count, plans, [&](int first, int cnt) -> edkm_status {
        BatchArgs b;
        std::memset(&b, 0, sizeof(b));
        b.count = cnt;
        bool vec = true;
        for (int i = 0; i < cnt; ++i) {
            const PlanImpl* P = impl(plans[first + i]);
            fill_mat(b.m[i], P, w_bits[first + i]);
            b.m[i].nuniq_out = num_unique_out ? num_unique_out[first + i] : nullptr;
            vec = vec && aligned16(w_bits[first + i]);
        }
        for (int i = 0; i < cnt; ++i) b.m[i].vec = vec;
        const uint32_t grid = partition(b, np_budget());
        const char* where = "";
        const hipError_t e = launch_init_unique(b, grid, stream, &where, &impl(plans[first])->ev);
        if (e != hipSuccess) return hip_fail(plans, first, cnt, e, where);
        return EDKM_OK;
    });
    if (st != EDKM_OK) return st;
    for (int i = 0; i < count; ++i) {
        if (counts_out && counts_out[i]) {
            Ws w = carve_workspace(impl(plans[i])->ws, impl(plans[i])->max_iter);
            const hipError_t e = hipMemcpyAsync(counts_out[i], w.counts, NKEYS * sizeof(uint32_t),
                                                hipMemcpyDeviceToDevice, stream);
            if (e != hipSuccess) return hip_fail(plans, i, 1, e, "hipMemcpyAsync(counts)");
        }
    }
    // As the single-matrix form on each: a matrix with non-finite weights
    // leaves its own plan uncounted, the others are counted.
    bool any_bad = false;
    for (int i = 0; i < count; ++i) {
        bool bad = false;
        if (check_finite) {
            Ws w = carve_workspace(impl(plans[i])->ws, impl(plans[i])->max_iter);
            uint32_t flag = 0;
            hipError_t e = hipMemcpyAsync(&flag, &w.st->nonfinite, sizeof(flag),
                                          hipMemcpyDeviceToHost, stream);
            if (e == hipSuccess) e = hipStreamSynchronize(stream);
            if (e != hipSuccess) return hip_fail(plans, i, 1, e, "non-finite check");
            bad = flag != 0;
        }
        PlanImpl* P = impl(plans[i]);
        P->stage = bad ? PLANNED : COUNTED;
        P->keys = bad ? nullptr : w_bits[i];
        any_bad = any_bad || bad;
    }
    return any_bad ? EDKM_ERR_NONFINITE : EDKM_OK;
}

edkm_status edkm_init_unique(edkm_plan* plan, const uint16_t* w_bits, uint32_t* counts_out,
                             uint32_t* num_unique_out, int check_finite, hipStream_t stream) {
    return edkm_init_unique_batch(1, &plan, &w_bits, &counts_out, &num_unique_out, check_finite,
                                  stream);
}

edkm_status edkm_forward_batch(int count, edkm_plan* const* plans, const uint16_t* const* w_bits,
                               float tau, float eps, const float* const* c_in,
                               float* const* c_out, void* const* w_tilde, int out_half,
                               int32_t* const* iters_out, hipStream_t stream) {
    edkm_status st = check_batch(count, plans, w_bits);
    if (st != EDKM_OK) return st;
    if (!tau_ok(tau) || !eps_ok(eps) || !c_in || !c_out || !w_tilde ||
        (out_half != 0 && out_half != 1))
        return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i)
        if (!c_in[i] || !c_out[i] || !w_tilde[i]) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i) {
        const PlanImpl* P = impl(plans[i]);
        if (P->stage < COUNTED || P->stage == DENSE_FORWARD || P->keys != w_bits[i])
            return EDKM_ERR_STATE;
    }
    // From the first launch on, the table state of an earlier forward is being
    // overwritten: until this call succeeds, a backward needs a new forward.
    for (int i = 0; i < count; ++i) impl(plans[i])->stage = COUNTED;
    st = for_groups(count, plans, [&](int first, int cnt) -> edkm_status {
        BatchArgs b;
        std::memset(&b, 0, sizeof(b));
        b.count = cnt;
        b.out_half = out_half;
        b.s2 = tau_s2(tau);
        b.inv_tau = 1.0f / tau;
        b.eps = eps;
        bool vec = true;
        int max_t = 0;
        for (int i = 0; i < cnt; ++i) {
            const int q = first + i;
            const PlanImpl* P = impl(plans[q]);
            MatArgs& M = b.m[i];
            fill_mat(M, P, w_bits[q]);
            M.c_in = c_in[q];
            M.c_out = c_out[q];
            M.wt = w_tilde[q];
            M.iters_out = iters_out ? iters_out[q] : nullptr;
            vec = vec && aligned16(w_bits[q]) && aligned16(w_tilde[q]);
            if (P->max_iter > max_t) max_t = P->max_iter;
        }
        for (int i = 0; i < cnt; ++i) b.m[i].vec = vec;
        const uint32_t grid = partition(b, np_budget());
        const char* where = "";
        const hipError_t e = launch_forward(b, grid, max_t, stream, &where, &impl(plans[first])->ev);
        if (e != hipSuccess) return hip_fail(plans, first, cnt, e, where);
        return EDKM_OK;
    });
    if (st != EDKM_OK) return st;
    for (int i = 0; i < count; ++i) {
        PlanImpl* P = impl(plans[i]);
        P->stage = FORWARD;
        P->tau = tau;
        P->eps = eps;
    }
    return EDKM_OK;
}

edkm_status edkm_forward(edkm_plan* plan, const uint16_t* w_bits, float tau, float eps,
                         const float* c_in, float* c_out, void* w_tilde, int out_half,
                         int32_t* iters_out, hipStream_t stream) {
    return edkm_forward_batch(1, &plan, &w_bits, tau, eps, &c_in, &c_out, &w_tilde, out_half,
                              &iters_out, stream);
}

edkm_status edkm_backward_batch_ex(int count, edkm_plan* const* plans, const uint16_t* const* w_bits,
                                   const void* const* grad_w_tilde, void* const* grad_w,
                                   float* const* grad_c, int flags, hipStream_t stream) {
    edkm_status st = check_batch(count, plans, w_bits);
    if (st != EDKM_OK) return st;
    if (flags & ~(EDKM_GRAD_IN_HALF | EDKM_GRAD_OUT_HALF)) return EDKM_ERR_ARG;
    if (!grad_w_tilde || !grad_w || !grad_c) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i)
        if (!grad_w_tilde[i] || !grad_w[i] || !grad_c[i]) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i) {
        const PlanImpl* P = impl(plans[i]);
        if (P->stage != FORWARD || P->keys != w_bits[i]) return EDKM_ERR_STATE;
    }
    // one tau per launch group: split groups where tau differs
    st = for_groups(count, plans, [&](int first, int cnt) -> edkm_status {
        int i0 = 0;
        while (i0 < cnt) {
            int i1 = i0 + 1;
            while (i1 < cnt && impl(plans[first + i1])->tau == impl(plans[first + i0])->tau) ++i1;
            BatchArgs b;
            std::memset(&b, 0, sizeof(b));
            b.count = i1 - i0;
            const float tau = impl(plans[first + i0])->tau;
            b.s2 = tau_s2(tau);
            b.inv_tau = 1.0f / tau;
            b.g_half = (flags & EDKM_GRAD_IN_HALF) != 0;
            b.gw_half = (flags & EDKM_GRAD_OUT_HALF) != 0;
            bool vec = true;
            int max_t = 0;
            for (int i = 0; i < b.count; ++i) {
                const int q = first + i0 + i;
                const PlanImpl* P = impl(plans[q]);
                MatArgs& M = b.m[i];
                fill_mat(M, P, w_bits[q]);
                M.g = static_cast<const float*>(grad_w_tilde[q]);   // 16-bit patterns with g_half
                M.gw = static_cast<float*>(grad_w[q]);              // 16-bit patterns with gw_half
                M.gc = grad_c[q];
                vec = vec && aligned16(w_bits[q]) && aligned16(grad_w_tilde[q]) &&
                      aligned16(grad_w[q]);
                if (P->max_iter > max_t) max_t = P->max_iter;
            }
            for (int i = 0; i < b.count; ++i) b.m[i].vec = vec;
            const uint32_t grid = partition(b, np_budget());
            const char* where = "";
            const hipError_t e =
                launch_backward(b, grid, max_t, stream, &where, &impl(plans[first + i0])->ev);
            if (e != hipSuccess) return hip_fail(plans, first + i0, b.count, e, where);
            i0 = i1;
        }
        return EDKM_OK;
    });
    if (st == EDKM_ERR_HIP) {
        // a backward that did not run to its end may leave its table partials
        // half-added: the next backward needs a new forward (which clears them)
        for (int i = 0; i < count; ++i) impl(plans[i])->stage = COUNTED;
    }
    return st;
}

edkm_status edkm_backward_batch(int count, edkm_plan* const* plans, const uint16_t* const* w_bits,
                                const float* const* grad_w_tilde, float* const* grad_w,
                                float* const* grad_c, hipStream_t stream) {
    return edkm_backward_batch_ex(count, plans, w_bits, reinterpret_cast<const void* const*>(grad_w_tilde),
                                  reinterpret_cast<void* const*>(grad_w), grad_c, 0, stream);
}

edkm_status edkm_backward(edkm_plan* plan, const uint16_t* w_bits, const float* grad_w_tilde,
                          float* grad_w, float* grad_c, hipStream_t stream) {
    return edkm_backward_batch(1, &plan, &w_bits, &grad_w_tilde, &grad_w, &grad_c, stream);
}

edkm_status edkm_backward_ex(edkm_plan* plan, const uint16_t* w_bits, const void* grad_w_tilde,
                             void* grad_w, float* grad_c, int flags, hipStream_t stream) {
    return edkm_backward_batch_ex(1, &plan, &w_bits, &grad_w_tilde, &grad_w, &grad_c, flags, stream);
}

edkm_status edkm_forward_dense(edkm_plan* plan, const uint16_t* w_bits, float tau, float eps,
                               const float* c_in, float* c_out, void* w_tilde, int out_half,
                               int32_t* iters_out, float* attn_out, hipStream_t stream) {
    if (!plan_ok(plan) || !w_bits || !tau_ok(tau) || !eps_ok(eps) || !c_in || !c_out ||
        !w_tilde || (out_half != 0 && out_half != 1))
        return EDKM_ERR_ARG;
    PlanImpl* P = impl(plan);
    BatchArgs b;
    std::memset(&b, 0, sizeof(b));
    b.count = 1;
    b.out_half = out_half;
    b.s2 = tau_s2(tau);
    b.inv_tau = 1.0f / tau;
    b.eps = eps;
    MatArgs& M = b.m[0];
    fill_mat(M, P, w_bits);
    M.c_in = c_in;
    M.c_out = c_out;
    M.wt = w_tilde;
    M.iters_out = iters_out;
    M.attn = attn_out;
    uint64_t nwg = (P->n + 4095) / 4096;
    if (nwg > (uint64_t)D_WG) nwg = D_WG;
    M.chunk = (P->n + nwg - 1) / nwg;
    // the dense kernels reuse the workspace's iteration history: whatever
    // state it held is gone once they launch, whether or not they succeed
    P->stage = PLANNED;
    P->keys = nullptr;
    const char* where = "";
    const hipError_t e = launch_forward_dense(b, (uint32_t)nwg, stream, &where, &P->ev);
    if (e != hipSuccess) return hip_fail(&plan, 0, 1, e, where);
    P->stage = DENSE_FORWARD;
    P->keys = w_bits;
    P->tau = tau;
    P->eps = eps;
    return EDKM_OK;
}

edkm_status edkm_backward_dense(edkm_plan* plan, const uint16_t* w_bits, const float* grad_w_tilde,
                                float* grad_w, float* grad_c, hipStream_t stream) {
    if (!plan_ok(plan) || !w_bits || !grad_w_tilde || !grad_w || !grad_c) return EDKM_ERR_ARG;
    PlanImpl* P = impl(plan);
    if (P->stage != DENSE_FORWARD || P->keys != w_bits) return EDKM_ERR_STATE;
    BatchArgs b;
    std::memset(&b, 0, sizeof(b));
    b.count = 1;
    b.s2 = tau_s2(P->tau);
    b.inv_tau = 1.0f / P->tau;
    MatArgs& M = b.m[0];
    fill_mat(M, P, w_bits);
    M.g = grad_w_tilde;
    M.gw = grad_w;
    M.gc = grad_c;
    uint64_t nwg = (P->n + 4095) / 4096;
    if (nwg > (uint64_t)D_WG) nwg = D_WG;
    M.chunk = (P->n + nwg - 1) / nwg;
    const char* where = "";
    const hipError_t e = launch_backward_dense(b, (uint32_t)nwg, stream, &where, &P->ev);
    if (e != hipSuccess) return hip_fail(&plan, 0, 1, e, where);
    return EDKM_OK;
}

edkm_status edkm_plan_set_pass_events(edkm_plan* plan, int pass, hipEvent_t start, hipEvent_t stop) {
    if (!plan_ok(plan) || pass < 0 || pass >= NPASS) return EDKM_ERR_ARG;
    PlanImpl* P = impl(plan);
    P->ev.start[pass] = start;
    P->ev.stop[pass] = stop;
    return EDKM_OK;
}

edkm_status edkm_palettize(edkm_plan* plan, const uint16_t* w_bits, const float* lut,
                           uint8_t* indices_out, hipStream_t stream) {
    return edkm_palettize_batch(1, &plan, &w_bits, &lut, &indices_out, stream);
}

edkm_status edkm_palettize_batch(int count, edkm_plan* const* plans, const uint16_t* const* w_bits,
                                 const float* const* lut, uint8_t* const* indices_out,
                                 hipStream_t stream) {
    edkm_status st = check_batch(count, plans, w_bits);
    if (st != EDKM_OK) return st;
    if (!lut || !indices_out) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i)
        if (!lut[i] || !indices_out[i]) return EDKM_ERR_ARG;
    return for_groups(count, plans, [&](int first, int cnt) -> edkm_status {
        BatchArgs b;
        std::memset(&b, 0, sizeof(b));
        b.count = cnt;
        for (int i = 0; i < cnt; ++i) {
            const int q = first + i;
            MatArgs& M = b.m[i];
            fill_mat(M, impl(plans[q]), w_bits[q]);
            M.c_in = lut[q];
            M.wt = indices_out[q];
            M.vec = aligned16(w_bits[q]) && ((uintptr_t)indices_out[q] & 3u) == 0;
        }
        // the packing kernel's 64 KiB index table leaves room for two workgroups per CU
        const uint32_t grid = partition(b, 2 * np_budget());
        const char* where = "";
        const hipError_t e = launch_palettize(b, grid, stream, &where, &impl(plans[first])->ev);
        if (e != hipSuccess) return hip_fail(plans, first, cnt, e, where);
        return EDKM_OK;
    });
}

edkm_status edkm_palettize_noalloc(const uint16_t* w_bits, uint64_t n, int bits, int key_format,
                                   const float* lut, uint8_t* indices_out, hipStream_t stream) {
    if (!w_bits || !lut || !indices_out || n < 1 || n > EDKM_MAX_N || bits < 1 ||
        bits > EDKM_MAX_BITS || (key_format != EDKM_KEYS_FP16 && key_format != EDKM_KEYS_BF16))
        return EDKM_ERR_ARG;
    uint8_t* tab = nullptr;
    if (noalloc_scratch(&tab) != hipSuccess) return EDKM_ERR_HIP;
    BatchArgs b;
    std::memset(&b, 0, sizeof(b));
    b.count = 1;
    b.pal_tab = tab;   // the library's array on this device: no workspace
    MatArgs& M = b.m[0];
    M.keys = w_bits;
    M.n = n;
    M.k = 1 << bits;
    M.max_iter = 1;
    M.fmt = key_format == EDKM_KEYS_BF16 ? FMT_BF16 : FMT_FP16;
    M.c_in = lut;
    M.wt = indices_out;
    M.vec = aligned16(w_bits) && ((uintptr_t)indices_out & 3u) == 0;
    // the packing kernel's 64 KiB index table leaves room for two workgroups per CU
    const uint32_t grid = partition(b, 2 * np_budget());
    const char* where = "";
    return launch_palettize(b, grid, stream, &where, nullptr) == hipSuccess ? EDKM_OK : EDKM_ERR_HIP;
}

edkm_status edkm_unique_inverse(edkm_plan* plan, const uint16_t* w_bits, uint16_t* unique_out,
                                uint16_t* inverse_out, hipStream_t stream) {
    return edkm_unique_inverse_batch(1, &plan, &w_bits, &unique_out, &inverse_out, stream);
}

edkm_status edkm_unique_inverse_batch(int count, edkm_plan* const* plans,
                                      const uint16_t* const* w_bits, uint16_t* const* unique_out,
                                      uint16_t* const* inverse_out, hipStream_t stream) {
    edkm_status st = check_batch(count, plans, w_bits);
    if (st != EDKM_OK) return st;
    auto uniq = [&](int i) { return unique_out ? unique_out[i] : nullptr; };
    auto inv = [&](int i) { return inverse_out ? inverse_out[i] : nullptr; };
    for (int i = 0; i < count; ++i)
        if (!uniq(i) && !inv(i)) return EDKM_ERR_ARG;
    for (int i = 0; i < count; ++i) {
        const PlanImpl* P = impl(plans[i]);
        if ((P->stage != COUNTED && P->stage != FORWARD) || P->keys != w_bits[i]) return EDKM_ERR_STATE;
    }
    return for_groups(count, plans, [&](int first, int cnt) -> edkm_status {
        BatchArgs b;
        std::memset(&b, 0, sizeof(b));
        b.count = cnt;
        bool vec = true, any_inv = false;
        for (int i = 0; i < cnt; ++i) {
            const int q = first + i;
            MatArgs& M = b.m[i];
            fill_mat(M, impl(plans[q]), w_bits[q]);
            M.uniq = uniq(q);
            M.wt = inv(q);
            any_inv = any_inv || M.wt;
            vec = vec && aligned16(w_bits[q]) && (!M.wt || aligned16(M.wt));
        }
        for (int i = 0; i < cnt; ++i) b.m[i].vec = vec;
        const uint32_t grid = partition(b, np_budget());
        const char* where = "";
        const hipError_t e =
            launch_unique_inverse(b, grid, any_inv, stream, &where, &impl(plans[first])->ev);
        if (e != hipSuccess) return hip_fail(plans, first, cnt, e, where);
        return EDKM_OK;
    });
}

edkm_status edkm_plan_set_keyed_mode(edkm_plan* plan, int mode) {
    if (!plan_ok(plan) || mode < EDKM_KEYED_AUTO || mode > EDKM_KEYED_U64) return EDKM_ERR_ARG;
    impl(plan)->kforce = mode;
    return EDKM_OK;
}

edkm_status edkm_plan_hip_error(const edkm_plan* plan, int* code, const char** step,
                                const char** message) {
    if (!plan_ok(plan)) return EDKM_ERR_ARG;
    const PlanImpl* P = reinterpret_cast<const PlanImpl*>(plan);
    if (code) *code = P->hip_code;
    if (step) *step = P->hip_step ? P->hip_step : "";
    if (message) *message = P->hip_code ? hipGetErrorString((hipError_t)P->hip_code) : "";
    return EDKM_OK;
}

const char* edkm_status_str(edkm_status s) {
    switch (s) {
    case EDKM_OK: return "ok";
    case EDKM_ERR_ARG: return "invalid argument";
    case EDKM_ERR_NONFINITE: return "non-finite weight (Inf or NaN)";
    case EDKM_ERR_WORKSPACE: return "workspace null, too small or not 256-byte aligned";
    case EDKM_ERR_STATE: return "call out of order for this plan, or a different key buffer";
    case EDKM_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

}  // extern "C"
