// Internal declarations shared by the eDKM kernels and the C-ABI layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "edkm.h"

namespace edkm {

constexpr int NKEYS = 65536;          // every 16-bit pattern
constexpr int MAGS = 0x8000;          // magnitudes (low 15 bits) of a 16-bit pattern
// Weight formats (the key is the raw 16-bit pattern either way).
constexpr int FMT_FP16 = 0;           // IEEE binary16: 5 exponent, 10 mantissa bits
constexpr int FMT_BF16 = 1;           // bfloat16: 8 exponent, 7 mantissa bits
// Magnitudes below this are finite in the format (above: Inf/NaN).
__host__ __device__ constexpr int fin_mags(int fmt) { return fmt == FMT_BF16 ? 0x7F80 : 0x7C00; }
constexpr int W4 = 19456;             // magnitudes per sign in a 4-byte LDS window (152 KiB)
constexpr int W8 = 10232;             // magnitudes per sign in the 8-byte LDS window (<160 KiB)
constexpr int NP_THREADS = 1024;      // N-pass workgroup size
constexpr int NP_MAX_WG = 256;        // N-pass workgroups per launch group, at most (one per CU)
constexpr int NP_MIN_CHUNK = 16384;   // smallest slice of a matrix given to one workgroup
constexpr int ROW4 = 2 * W4;          // 32-bit words per N-pass partial row
constexpr int T_WG = 64;              // table-phase workgroups per matrix (a multiple of 64)
constexpr int T_THREADS = 256;
constexpr int T_KPT = NKEYS / (T_WG * T_THREADS);   // patterns per table-phase thread
constexpr int KMAX = 16;
constexpr int PSTRIDE = 32;           // floats per table-phase partial row (2 * KMAX)
constexpr int MAXB = EDKM_LAUNCH_GROUP;   // matrices per launch
constexpr int D_WG = 1024;            // dense path: max workgroups
constexpr int D_THREADS = 256;

// Device-side per-matrix state (in the workspace).
struct DevState {
    int teff;            // iterations executed by the last forward
    int conv;            // 1 once the eps criterion stopped the iteration
    uint32_t nonfinite;  // 1 if any weight is Inf/NaN
    uint32_t num_unique; // occupied patterns
    int lo4, w4;         // 4-byte table window: magnitudes [lo4, lo4 + w4), both signs
    int lo8, w8;         // 8-byte table window
    int mlo, mhi;        // occupied finite magnitude range
    int kmode;           // keyed-sum accumulators: KEYED_I32 or KEYED_U64 (chosen by k_window)
    int pad[5];
};

// Device pointers into one plan's workspace.
struct Ws {
    uint32_t* counts;   // [NKEYS]
    float* tab;         // [NKEYS]  W~ value per pattern
    float* H;           // [NKEYS]  dW~/dw per pattern (through the final softmax)
    float* R;           // [NKEYS]  accumulated R during the backward
    float2* HR;         // [NKEYS]  (H, R) for the gradient gather
    float* G;           // [NKEYS]  keyed gradient sums outside the LDS window
    float* chist;       // [(max_iter+1) * KMAX]  C^(t)
    float* shist;       // [(max_iter+1) * KMAX]  S^(t)
    float* ghist;       // [(max_iter+1) * KMAX]  dL/dC^(t)
    float* ehist;       // [KMAX]  direct-use term of the dense backward
    float* cfin;        // [2 * KMAX]  C^(T-1), C^(T) of the last forward (at a fixed place)
    float* tpart;       // [(max_iter+1) * T_WG * PSTRIDE]  forward table partials
    float* bpart;       // [(max_iter+1) * T_WG * PSTRIDE]  backward table partials
    float* dpart;       // [D_WG * PSTRIDE]  dense-path partials
    int2* span;         // [NP_MAX_WG]  histogram partial spans
    uint32_t* part;     // [NP_MAX_WG * ROW4]  N-pass partial rows
    uint8_t* pidx;      // [NKEYS]  palettization: nearest lookup-table entry per pattern
    uint16_t* rank;     // [NKEYS]  occupied patterns below each pattern (unique_inverse)
    DevState* st;
};

// Keyed-sum accumulator modes (see k_keyed_grad).
constexpr int KEYED_I32 = 0;          // 32-bit, returning atomics, 4-byte window
constexpr int KEYED_U64 = 1;          // 64-bit, plain atomics, 8-byte window
// Switch to KEYED_U64 above this expected number of other lanes sharing an
// address per 64-lane atomic, 2016 sum_u (n_u / N)^2.
constexpr double KEYED_U64_ABOVE = 0.6;

// Everything a kernel needs about one matrix.
struct MatArgs {
    const uint16_t* keys;
    uint64_t n;
    const float* c_in;
    float* c_out;
    void* wt;                 // W~ output (float or 16-bit); packed indices (palettize);
                              // inverse index (unique_inverse)
    int32_t* iters_out;
    uint32_t* nuniq_out;
    const float* g;           // dL/dW~ (16-bit patterns when the launch's g_half is set)
    float* gw;                // dL/dw (16-bit patterns when the launch's gw_half is set)
    float* gc;                // dL/dC^(0)
    float* attn;              // dense map output (nullable)
    uint16_t* uniq;           // sorted distinct patterns (unique_inverse, nullable)
    void* wsb;                // workspace base (regions: carve_workspace)
    int k;
    int max_iter;
    uint64_t chunk;           // weights per N-pass workgroup (multiple of 8)
    int vec;                  // all N-sized buffers 16-byte aligned
    int fmt;                  // FMT_FP16 or FMT_BF16 (the same within a launch group)
    int kforce;               // keyed-sum mode forced by the caller, or -1 (chosen from the data)
    uint32_t wg_count;        // N-pass workgroups (= partial rows)
};

struct BatchArgs {
    int count;
    int t;                    // iteration index of a per-iteration launch
    int out_half;             // W~ as 16-bit floats of the weight format
    int g_half;               // dL/dW~ given as 16-bit floats of the weight format
    int gw_half;              // dL/dw written as 16-bit floats of the weight format
    float s2;                 // log2(e) / tau
    float inv_tau;
    float eps;
    float keep_frac;          // fraction of each sweep read with cached loads (its end)
#ifdef EDKM_BLOCK_STAMPS
    int stamp_slot;           // launch index in the stamp record (diagnostics build)
#endif
    uint8_t* pal_tab;         // palettization index table of the launch's single matrix
                              // (allocation-free entry point); null: each matrix's workspace
    // First N-pass workgroup of each matrix, ascending; 0xFFFFFFFF past the
    // launch's matrices.  Kept together (not in MatArgs) so that a workgroup
    // finds its matrix from contiguous scalar loads issued together instead
    // of 27 scattered ones (about 2 us per launch).
    uint32_t wg_begin[MAXB];
    MatArgs m[MAXB];
};

// Kernel arguments are passed by value; the launch limit is 4 KiB.
static_assert(sizeof(BatchArgs) <= 4096, "launch arguments fit the kernel-argument limit");

// Workspace layout: byte offsets of every region, each 256-byte aligned.  A
// function of max_iter only, evaluated on the host (sizing, plan checks) and
// in every kernel (from the workspace base in the launch arguments).
struct Layout {
    size_t counts, tab, H, R, HR, G, chist, shist, ghist, ehist, cfin, tpart, bpart, dpart, span, part, pidx,
        rank, st, total;
};

__host__ __device__ inline Layout layout(int max_iter) {
    Layout L{};
    size_t o = 0;
    auto take = [&](size_t bytes) { size_t at = o; o = (o + bytes + 255) & ~size_t(255); return at; };
    const size_t hist = (size_t)(max_iter + 1) * KMAX * sizeof(float);
    const size_t tp = (size_t)(max_iter + 1) * T_WG * PSTRIDE * sizeof(float);
    L.st = take(sizeof(DevState));
    L.counts = take(NKEYS * sizeof(uint32_t));
    L.tab = take(NKEYS * sizeof(float));
    L.H = take(NKEYS * sizeof(float));
    L.R = take(NKEYS * sizeof(float));
    L.HR = take(NKEYS * sizeof(float2));
    L.G = take(NKEYS * sizeof(float));
    L.chist = take(hist);
    L.shist = take(hist);
    L.ghist = take(hist);
    L.ehist = take(KMAX * sizeof(float));
    L.cfin = take(2 * KMAX * sizeof(float));
    L.tpart = take(tp);
    L.bpart = take(tp);
    L.dpart = take((size_t)D_WG * PSTRIDE * sizeof(float));
    L.span = take(NP_MAX_WG * sizeof(int2));
    L.part = take((size_t)NP_MAX_WG * ROW4 * sizeof(uint32_t));
    L.pidx = take(NKEYS);
    L.rank = take(NKEYS * sizeof(uint16_t));
    L.total = o;
    return L;
}

inline size_t workspace_bytes(int max_iter) { return layout(max_iter).total; }

__host__ __device__ inline Ws carve_workspace(void* base, int max_iter) {
    const Layout L = layout(max_iter);
    char* c = static_cast<char*>(base);
    Ws w;
    w.pidx = reinterpret_cast<uint8_t*>(c + L.pidx);
    w.rank = reinterpret_cast<uint16_t*>(c + L.rank);
    w.st = reinterpret_cast<DevState*>(c + L.st);
    w.counts = reinterpret_cast<uint32_t*>(c + L.counts);
    w.tab = reinterpret_cast<float*>(c + L.tab);
    w.H = reinterpret_cast<float*>(c + L.H);
    w.R = reinterpret_cast<float*>(c + L.R);
    w.HR = reinterpret_cast<float2*>(c + L.HR);
    w.G = reinterpret_cast<float*>(c + L.G);
    w.chist = reinterpret_cast<float*>(c + L.chist);
    w.shist = reinterpret_cast<float*>(c + L.shist);
    w.ghist = reinterpret_cast<float*>(c + L.ghist);
    w.ehist = reinterpret_cast<float*>(c + L.ehist);
    w.cfin = reinterpret_cast<float*>(c + L.cfin);
    w.tpart = reinterpret_cast<float*>(c + L.tpart);
    w.bpart = reinterpret_cast<float*>(c + L.bpart);
    w.dpart = reinterpret_cast<float*>(c + L.dpart);
    w.span = reinterpret_cast<int2*>(c + L.span);
    w.part = reinterpret_cast<uint32_t*>(c + L.part);
    return w;
}

// Optional timing events recorded around the N-sized passes (diagnostics).
enum Pass { PASS_HIST = 0, PASS_GATHER_WT = 1, PASS_KEYED_GRAD = 2, PASS_GATHER_GRAD = 3,
            PASS_DENSE_ITER = 4, PASS_DENSE_BITER = 5, PASS_PALETTIZE = 6, PASS_INVERSE = 7,
            NPASS = 8 };
struct PassEvents {
    hipEvent_t start[NPASS];
    hipEvent_t stop[NPASS];
};


// The allocation-free palettization keeps its index table (one byte per
// pattern) in a library-owned device array of this size, one per GPU.
constexpr size_t NOALLOC_SCRATCH_BYTES = NKEYS;
// Address of that array on the current device (looked up once per device).
hipError_t noalloc_scratch(uint8_t** out);

// Launch sequences (all asynchronous on `s`).  Each returns the first HIP error.
// On failure *where names the launch that failed.
hipError_t launch_init_unique(BatchArgs& b, uint32_t grid_np, hipStream_t s, const char** where,
                              const PassEvents* ev = nullptr);
hipError_t launch_forward(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                              const PassEvents* ev = nullptr);
hipError_t launch_backward(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                              const PassEvents* ev = nullptr);
hipError_t launch_palettize(BatchArgs& b, uint32_t grid_np, hipStream_t s, const char** where,
                            const PassEvents* ev);
hipError_t launch_unique_inverse(BatchArgs& b, uint32_t grid_np, bool inverse, hipStream_t s,
                                 const char** where, const PassEvents* ev);
hipError_t launch_forward_dense(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                const PassEvents* ev = nullptr);
hipError_t launch_backward_dense(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                 const PassEvents* ev = nullptr);

}  // namespace edkm
