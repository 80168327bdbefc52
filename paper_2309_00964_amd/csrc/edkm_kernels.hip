// eDKM hot-path kernels for gfx950 (MI355X).
//
// Uniquified DKM (paper Sec. 2.2): the attention map of N 16-bit weights (fp16
// or bf16) against k <= 16 centroids is kept as a 65,536-row table indexed by
// the weights' own bit patterns.  Work splits into
//   * N-sized passes, bound by HBM bandwidth: the pattern histogram, the W~
//     gather, the keyed reduction of dL/dW~ and the dL/dw gather.  They run one
//     1024-thread workgroup per CU, keep a window of the table in LDS (up to
//     160 KiB), sweep each matrix in round-robin tiles with vector loads and
//     merge per-workgroup results through dense partial rows instead of global
//     atomics;
//   * table-sized phases, bound by latency: the T softmax / centroid-update
//     iterations and the unrolled analytic backward, one launch per iteration,
//     64 workgroups per matrix, fixed-order tree reductions so the forward is
//     bitwise repeatable;
//   * the dense comparison path (the same mathematics per weight over the
//     N x k map) and the palettization export (packed nearest-entry indices).
// Every launch carries up to MAXB = 28 matrices (blockIdx.y or a workgroup
// range per matrix), so a decoder layer, or four of them, pays each launch
// latency once.
//
// Nothing here uses MFMA: k <= 16 centroids is not a dense contraction.

#include "edkm_internal.h"
#ifdef EDKM_BLOCK_STAMPS
#include "edkm_stamps.h"
#endif

#include <hip/hip_fp16.h>
#include <algorithm>
#include <atomic>

namespace edkm {

// ----------------------------------------------------------------------------
// Block timeline (diagnostics build only, -DEDKM_BLOCK_STAMPS): thread 0 of
// every block records the wall clock (s_memrealtime, 100 MHz) at entry and the
// block's XCC id, each wave's lane 0 raises the block's end stamp as it
// leaves, and a few kernels stamp the phases of their block
// (EDKM_STAMP_MARK).  Launches are numbered in enqueue order from the last
// edkm_stamps_reset(); the first STAMP_LAUNCHES launches and STAMP_BLOCKS
// blocks of each are kept.  The product build compiles none of this.
#ifdef EDKM_BLOCK_STAMPS
constexpr int STAMP_LAUNCHES = EDKM_STAMP_LAUNCHES, STAMP_BLOCKS = EDKM_STAMP_BLOCKS,
              STAMP_WORDS = EDKM_STAMP_WORDS;
__device__ unsigned long long stamp_ts[STAMP_LAUNCHES * STAMP_BLOCKS * STAMP_WORDS];
__device__ __forceinline__ unsigned long long* stamp_row(int slot) {
    const unsigned lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    if (slot < 0 || slot >= STAMP_LAUNCHES || lin >= STAMP_BLOCKS) return nullptr;
    return stamp_ts + ((size_t)slot * STAMP_BLOCKS + lin) * STAMP_WORDS;
}
struct StampScope {   // words: 0 entry, 1 end, 2..6 phase marks, 7 XCC id
    int slot;
    __device__ explicit StampScope(int s) : slot(s) {
        unsigned long long* r = stamp_row(slot);
        if (r && threadIdx.x == 0) {
            r[0] = wall_clock64();
            unsigned x;
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
            r[7] = x;
        }
    }
    __device__ ~StampScope() {
        unsigned long long* r = stamp_row(slot);
        if (r && (threadIdx.x & 63) == 0) atomicMax(r + 1, wall_clock64());
    }
};
#define EDKM_STAMP_ENTRY(b) StampScope stamp_scope_((b).stamp_slot)
#define EDKM_STAMP_MARK(b, i)                                                         \
    do {                                                                              \
        unsigned long long* r_ = stamp_row((b).stamp_slot);                           \
        if (r_ && threadIdx.x == 0) r_[i] = wall_clock64();                           \
    } while (0)
static int g_stamp_seq = 0;
static char g_stamp_names[STAMP_LAUNCHES][32];
static int stamp_next(const char* name) {
    const int q = g_stamp_seq++;
    if (q >= STAMP_LAUNCHES) return -1;
    for (int i = 0; i < 31; ++i) { g_stamp_names[q][i] = name[i]; if (!name[i]) break; }
    g_stamp_names[q][31] = 0;
    return q;
}
#define EDKM_STAMP_SLOT(b, name) ((b).stamp_slot = stamp_next(name))
#else
#define EDKM_STAMP_ENTRY(b) ((void)0)
#define EDKM_STAMP_MARK(b, i) ((void)0)
#define EDKM_STAMP_SLOT(b, name) ((void)0)
#endif

// ----------------------------------------------------------------------------
// small device helpers

// 16-bit pattern -> fp32, exact for finite values including subnormals.
// fp16: integer decode, independent of the denormal mode.  bf16: the upper
// half of the binary32 pattern; its subnormals are fp32 subnormals, which the
// kernels keep (fp32 denormal mode "preserve", the HIP default).
__device__ __forceinline__ float key_value(uint32_t h, int fmt) {
    if (fmt == FMT_BF16) return __uint_as_float(h << 16);
    const uint32_t e = (h >> 10) & 0x1Fu;
    const uint32_t m = h & 0x3FFu;
    float mag = e ? __uint_as_float(((e + 112u) << 23) | (m << 13)) : (float)m * 0x1p-24f;
    return __uint_as_float(__float_as_uint(mag) | ((h & 0x8000u) << 16));
}

__device__ __forceinline__ bool key_finite(uint32_t h, int fmt) {
    return (int)(h & 0x7FFFu) < fin_mags(fmt);
}

// 16-bit gradient value -> fp32, exact, Inf and NaN included (unlike
// key_value, which only ever sees finite patterns).
__device__ __forceinline__ float grad_value(uint32_t h, int fmt) {
    if (fmt == FMT_BF16) return __uint_as_float(h << 16);
    return __half2float(__ushort_as_half((unsigned short)h));
}

// fp32 -> 16-bit pattern of the weight format, round to nearest even (NaN
// stays NaN).
__device__ __forceinline__ uint32_t to_half_bits(float x, int fmt) {
    if (fmt == FMT_FP16) return (uint32_t)__half_as_ushort(__float2half_rn(x));
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float sgnf(float x) { return (float)((x > 0.f) - (x < 0.f)); }

// One attention row: a_j = softmax_j(-|v - c_j| / tau), with s2 = log2(e) / tau.
// m is the nearest centroid; attn_row_sel also returns e[m] for a companion
// array e.  The exponent -(|v - c_j| - |v - c_m|) / tau
// is formed without subtracting two distances of size |v|: when v lies on the
// same side of c_j and c_m the difference is exactly |c_j - c_m|, otherwise v
// lies between them and both distances are at most |c_j - c_m|.  (Subtracting
// fp32 distances directly loses every digit once |v| is large against the
// centroid spacing, e.g. an outlier far from the bulk.)
template <int K>
__device__ __forceinline__ void attn_row_sel(float v, const float (&c)[K], float s2, float (&a)[K],
                                             const float (&e)[K], float& em) {
    float t[K];
#pragma unroll
    for (int j = 0; j < K; ++j) t[j] = v - c[j];
    // nearest centroid (first on ties), tracked by value: no run-time index
    float xm = fabsf(t[0]), cm = c[0], tm = t[0];
    em = e[0];
#pragma unroll
    for (int j = 1; j < K; ++j) {
        if (fabsf(t[j]) < xm) { xm = fabsf(t[j]); cm = c[j]; tm = t[j]; em = e[j]; }
    }
    const uint32_t sm = __float_as_uint(tm) >> 31;
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const bool same = (__float_as_uint(t[j]) >> 31) == sm;
        const float d = same ? fabsf(c[j] - cm) : fabsf(t[j]) - xm;
        a[j] = __builtin_amdgcn_exp2f(-d * s2);
        sum += a[j];
    }
    const float r = 1.0f / sum;
#pragma unroll
    for (int j = 0; j < K; ++j) a[j] *= r;
}

template <int K>
__device__ __forceinline__ void attn_row(float v, const float (&c)[K], float s2, float (&a)[K]) {
    float unused;
    attn_row_sel<K>(v, c, s2, a, c, unused);
}

// Attention row of the dense comparison path.  The exponent is formed from
// plain fp32 distances, -(|v - c_j| - x) with x = min_i |v - c_i|, at about a
// third of attn_row_sel's instructions.  Each distance carries a rounding
// error of at most 2^-24 of itself, so for every a_j >= 2^-24 the exponent is
// off by at most about (x s2 + 24) 2^-24 (in units of log2).  The row is used
// while x s2 <= DENSE_FAST_X (a_j within 1.2e-5 relative); a weight farther
// than that from every centroid (a far outlier) takes attn_row_sel.  e and em
// as in attn_row_sel (nearest centroid, first on ties).
constexpr float DENSE_FAST_X = 256.f;

// Unnormalised form: a_j up to the factor r it returns (r = 1 after the
// careful row, which normalises itself).
template <int K>
__device__ __forceinline__ float attn_row_dense_un(float v, const float (&c)[K], float s2, float (&a)[K],
                                                   const float (&e)[K], float& em) {
    float d[K];
    d[0] = fabsf(v - c[0]);
    float xm = d[0];
    em = e[0];
#pragma unroll
    for (int j = 1; j < K; ++j) {
        d[j] = fabsf(v - c[j]);
        if (d[j] < xm) { xm = d[j]; em = e[j]; }
    }
    const float off = xm * s2;
    if (off <= DENSE_FAST_X) {
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            a[j] = __builtin_amdgcn_exp2f(fmaf(-d[j], s2, off));
            sum += a[j];
        }
        return 1.0f / sum;
    }
    attn_row_sel<K>(v, c, s2, a, e, em);
    return 1.0f;
}

template <int K>
__device__ __forceinline__ void attn_row_dense(float v, const float (&c)[K], float s2, float (&a)[K],
                                               const float (&e)[K], float& em) {
    const float r = attn_row_dense_un<K>(v, c, s2, a, e, em);
#pragma unroll
    for (int j = 0; j < K; ++j) a[j] *= r;
}

// Deviations d_j = C^(T)_j - W~ of one map row a, W~ = sum_j a_j C^(T)_j,
// written around c1m = C^(T)_m of the nearest centroid m:
//   d_j = (C_j - c1m) - sum_i a_i (C_i - c1m),   W~ = c1m + sum_i a_i (C_i - c1m).
// For a nearly one-hot row the d_j are tiny; forming W~ first and subtracting
// it would leave them with the rounding error of W~ (one ulp of |C|), which
// the direct derivative -(1/tau) sum_j a_j d_j sgn(v - C^(T-1)_j) multiplies
// into every dL/dw_i of the pattern.  Returns W~.
template <int K>
__device__ __forceinline__ float centroid_dev(const float (&a)[K], const float (&c1)[K], float c1m,
                                              float (&d)[K]) {
    float dt = 0.f;
#pragma unroll
    for (int j = 0; j < K; ++j) dt = fmaf(a[j], c1[j] - c1m, dt);
#pragma unroll
    for (int j = 0; j < K; ++j) d[j] = (c1[j] - c1m) - dt;
    return c1m + dt;
}

// Softmax-Jacobian deviations of one table row in the backward:
//   dev_j = alpha_j - sum_i a_i alpha_i,  alpha_j = gS_j (v - c1_j),
// written around the reference cm = c1_m (m the nearest centroid) as
//   dev_j = (gS_j - gbar)(v - cm) - (gS_j (c1_j - cm) - hb),
//   gbar = sum_i a_i gS_i,  hb = sum_i a_i gS_i (c1_i - cm),
// which never subtracts two terms of size |v|.  Returns gbar.
template <int K>
__device__ __forceinline__ float softmax_dev(float v, const float (&a)[K], const float (&gS)[K],
                                             const float (&c1)[K], float cm, float (&dev)[K]) {
    float gbar = 0.f, hb = 0.f;
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const float ag = a[j] * gS[j];
        gbar += ag;
        hb = fmaf(ag, c1[j] - cm, hb);
    }
    const float w1 = v - cm;
#pragma unroll
    for (int j = 0; j < K; ++j) dev[j] = fmaf(gS[j] - gbar, w1, -fmaf(gS[j], c1[j] - cm, -hb));
    return gbar;
}

// DPP lane moves: a VALU operand read from another lane of the same row of 16
// lanes or, for the two broadcasts, from lane 15 of the row below / lane 31.
// Lanes outside row_mask keep `old`.  (__shfl_xor compiles to LDS-crossbar
// reads, one round trip per butterfly level: about 40% of a table kernel's
// time went there.)
constexpr int DPP_XOR1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <- lane 7 - i within each 8
constexpr int DPP_MIRROR = 0x140;       // lane i <- lane 15 - i within each row
constexpr int DPP_BCAST15 = 0x142;      // row r <- lane 15 of row r - 1
constexpr int DPP_BCAST31 = 0x143;      // rows 2, 3 <- lane 31
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ float dpp_f(float old, float x) {
    return __int_as_float(
        __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(x), CTRL, ROW_MASK, 0xF, false));
}

// Sum over the 64 lanes of a wave (all active), in a fixed association
// order: pairs, quads, eights and rows of 16 by DPP, then row 1 += row 0,
// row 3 += row 2, row 3 += rows 0-1; the total is lane 63's, returned to
// every lane.
__device__ __forceinline__ float wave_sum(float x) {
    x += dpp_f<DPP_XOR1>(x, x);
    x += dpp_f<DPP_XOR2>(x, x);
    x += dpp_f<DPP_HALF_MIRROR>(x, x);
    x += dpp_f<DPP_MIRROR>(x, x);
    x += dpp_f<DPP_BCAST15, 0xA>(0.f, x);
    x += dpp_f<DPP_BCAST31, 0xC>(0.f, x);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ int dpp_i(int old, int x) {
    return __builtin_amdgcn_update_dpp(old, x, CTRL, ROW_MASK, 0xF, false);
}
constexpr int DPP_SHR1 = 0x111, DPP_SHR2 = 0x112, DPP_SHR4 = 0x114, DPP_SHR8 = 0x118;   // lane i <- i - n in its row

// Inclusive prefix sum over the 64 lanes (all active): within rows of 16 by
// shifts of 1, 2, 4, 8 (lanes without a source add 0), then the row totals.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
    int v = (int)x;
    v += dpp_i<DPP_SHR1>(0, v);
    v += dpp_i<DPP_SHR2>(0, v);
    v += dpp_i<DPP_SHR4>(0, v);
    v += dpp_i<DPP_SHR8>(0, v);
    v += dpp_i<DPP_BCAST15, 0xA>(0, v);
    v += dpp_i<DPP_BCAST31, 0xC>(0, v);
    return (uint32_t)v;
}

// Reduction of a 32-bit integer over the 64 lanes (all active) by an
// associative, commutative op with identity id; every lane gets the result.
template <class Op>
__device__ __forceinline__ int wave_reduce(int x, int id, Op op) {
    x = op(x, dpp_i<DPP_XOR1>(x, x));
    x = op(x, dpp_i<DPP_XOR2>(x, x));
    x = op(x, dpp_i<DPP_HALF_MIRROR>(x, x));
    x = op(x, dpp_i<DPP_MIRROR>(x, x));
    x = op(x, dpp_i<DPP_BCAST15, 0xA>(id, x));
    x = op(x, dpp_i<DPP_BCAST31, 0xC>(id, x));
    return __builtin_amdgcn_readlane(x, 63);
}

// Sum of a 64-bit integer over the 64 lanes (all active); both halves move
// with the same lane pattern.
template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long old, unsigned long long x) {
    const uint32_t lo = (uint32_t)dpp_i<CTRL, ROW_MASK>((int)(uint32_t)old, (int)(uint32_t)x);
    const uint32_t hi = (uint32_t)dpp_i<CTRL, ROW_MASK>((int)(uint32_t)(old >> 32), (int)(uint32_t)(x >> 32));
    return ((unsigned long long)hi << 32) | lo;
}
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long x) {
    x += dpp_u64<DPP_XOR1>(x, x);
    x += dpp_u64<DPP_XOR2>(x, x);
    x += dpp_u64<DPP_HALF_MIRROR>(x, x);
    x += dpp_u64<DPP_MIRROR>(x, x);
    x += dpp_u64<DPP_BCAST15, 0xA>(0ull, x);
    x += dpp_u64<DPP_BCAST31, 0xC>(0ull, x);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
    return ((unsigned long long)hi << 32) | lo;
}
// Fill an LDS table: dst[i] = src[idx(i)] for i < n (n <= MAXN), by a block of
// NT threads.  Every load of a thread is issued before its first LDS write;
// written as a plain loop, each iteration waited for its load, so the copy
// cost one L2 round trip per iteration.  The caller synchronises the block.
template <int MAXN, int NT, class T, class Idx>
__device__ __forceinline__ void fill_lds(T* dst, const T* src, int n, Idx idx) {
    constexpr int PER = (MAXN + NT - 1) / NT;
    T v[PER];
#pragma unroll
    for (int c = 0; c < PER; ++c) {
        const int i = threadIdx.x + c * NT;
        if (i < n) v[c] = src[idx(i)];
    }
#pragma unroll
    for (int c = 0; c < PER; ++c) {
        const int i = threadIdx.x + c * NT;
        if (i < n) dst[i] = v[c];
    }
}

// Maximum of a 64-bit unsigned integer over the 64 lanes (all active).
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long x) {
    auto mx = [](unsigned long long a, unsigned long long b) { return a > b ? a : b; };
    x = mx(x, dpp_u64<DPP_XOR1>(x, x));
    x = mx(x, dpp_u64<DPP_XOR2>(x, x));
    x = mx(x, dpp_u64<DPP_HALF_MIRROR>(x, x));
    x = mx(x, dpp_u64<DPP_MIRROR>(x, x));
    x = mx(x, dpp_u64<DPP_BCAST15, 0xA>(0ull, x));
    x = mx(x, dpp_u64<DPP_BCAST31, 0xC>(0ull, x));
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
    return ((unsigned long long)hi << 32) | lo;
}
__device__ __forceinline__ int op_min(int a, int b) { return min(a, b); }
__device__ __forceinline__ int op_max(int a, int b) { return max(a, b); }
__device__ __forceinline__ int op_add(int a, int b) { return a + b; }
__device__ __forceinline__ int op_or(int a, int b) { return a | b; }

// Sum NV per-thread values over a block of NT threads into out[0..NV) (LDS),
// in a fixed order.  `scratch` holds NT/64 * NV floats.
template <int NV, int NT>
__device__ __forceinline__ void block_sum(const float (&v)[NV], float* scratch, float* out) {
    constexpr int NW = NT / 64;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        float s = wave_sum(v[j]);
        if (lane == 0) scratch[wave * NV + j] = s;
    }
    __syncthreads();
    if (threadIdx.x < NV) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) s += scratch[w * NV + threadIdx.x];
        out[threadIdx.x] = s;
    }
    __syncthreads();
}

// Rows lane, lane + 64, ... of column col of a table partial block (T_WG x
// PSTRIDE floats), summed in that order (one lane per 64 rows).
__device__ __forceinline__ float tpart_rows(const float* part, int lane, int col) {
    float x = part[lane * PSTRIDE + col];
#pragma unroll
    for (int q = 1; q < T_WG / 64; ++q) x += part[(lane + 64 * q) * PSTRIDE + col];
    return x;
}

// Pairwise (tree-shaped) sum of N values, N a power of two: neighbours first,
// (0 1) (2 3) ..., then (0..1 2..3) ..., so that sums taken level by level
// over the bits of an index, low bits first, form one binary tree over it.
template <int N>
__device__ __forceinline__ float tree_sum(float (&x)[N]) {
    static_assert(N >= 1 && (N & (N - 1)) == 0, "N: a power of two");
#pragma unroll
    for (int h = 1; h < N; h *= 2)
#pragma unroll
        for (int q = 0; q < N; q += 2 * h) x[q] += x[q + h];
    return x[0];
}

// Column totals of a table partial block (T_WG rows, PSTRIDE floats apart), in
// a fixed tree order and with every load issued up front: virtual column c of
// NC (a power of two, 4 <= NC <= T_THREADS) is read from src(c), a pointer to
// its row 0 (null: a column not read).  Thread t holds rows [R s, R s + R) of
// column c = t % NC, s = t / NC, R = T_WG NC / T_THREADS; stage() sums them
// pairwise into red[t] (T_THREADS floats of LDS) and synchronises the block;
// total(red, c) then sums the T_THREADS / NC segment sums of column c
// pairwise.  (Wave reductions per column had each cost a chain of dependent
// lane moves, and a kernel read its partial block only after its flags: two
// round trips to memory and about 2 us per table launch.)
template <int NC>
struct PartCols {
    static_assert(NC >= 4 && NC <= T_THREADS && (NC & (NC - 1)) == 0, "NC: a power of two in [4, T_THREADS]");
    static constexpr int SEGS = T_THREADS / NC;
    static constexpr int R = T_WG / SEGS;
    static_assert(R >= 1, "at least one row per thread");
    float x[R];
    template <class Src>
    __device__ __forceinline__ void load(Src src) {
        const int c = threadIdx.x % NC, sg = threadIdx.x / NC;
        const float* p = src(c);
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = p ? p[(size_t)(sg * R + r) * PSTRIDE] : 0.f;
    }
    // column c of the block at base (no null test, so no branch among the loads)
    __device__ __forceinline__ void load_block(const float* base) {
        const int c = threadIdx.x % NC, sg = threadIdx.x / NC;
        const float* p = base + c;
#pragma unroll
        for (int r = 0; r < R; ++r) x[r] = p[(size_t)(sg * R + r) * PSTRIDE];
    }
    __device__ __forceinline__ void stage(float* red) {
        red[threadIdx.x] = tree_sum<R>(x);
        __syncthreads();
    }
    __device__ __forceinline__ static float total(const float* red, int c) {
        float y[SEGS];
#pragma unroll
        for (int sg = 0; sg < SEGS; ++sg) y[sg] = red[sg * NC + c];
        return tree_sum<SEGS>(y);
    }
};

// Sum of NV per-thread values (NV a power of two dividing T_THREADS) over a
// T_THREADS block, in a fixed tree order: thread NV s + j sums value j of
// threads NV s .. NV s + NV - 1 pairwise, then thread j sums the T_THREADS /
// NV segment sums pairwise.  Returns the total of value threadIdx.x in threads
// [0, NV).  red: BLOCK_TOTAL_LDS(NV) floats of LDS; every thread
// calls it.  (One dependent chain of lane moves per value had cost 0.8-2.5 us
// per table kernel.)
#define BLOCK_TOTAL_LDS(NV) (T_THREADS * ((NV) + 1) + T_THREADS)
template <int NV>
__device__ __forceinline__ float block_total(const float (&v)[NV], float* red) {
    static_assert(NV <= T_THREADS && T_THREADS % NV == 0, "NV divides the block");
    constexpr int LD = NV + 1;   // odd pitch: a value's rows fall in different banks
    float* seg = red + T_THREADS * LD;
#pragma unroll
    for (int j = 0; j < NV; ++j) red[threadIdx.x * LD + j] = v[j];
    __syncthreads();
    const int j = threadIdx.x % NV, sg = threadIdx.x / NV;
    float a[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) a[i] = red[(sg * NV + i) * LD + j];
    seg[threadIdx.x] = tree_sum<NV>(a);
    __syncthreads();
    float tot = 0.f;
    if (threadIdx.x < NV) {
        float y[T_THREADS / NV];
#pragma unroll
        for (int q = 0; q < T_THREADS / NV; ++q) y[q] = seg[q * NV + threadIdx.x];
        tot = tree_sum<T_THREADS / NV>(y);
    }
    return tot;
}

// Matrix of an N-pass workgroup, and its slice [beg, end).
__device__ __forceinline__ int np_matrix(const BatchArgs& b) {
    // wg_begin ascends with the matrix (entries past the launch's matrices hold
    // 0xFFFFFFFF): count the matrices starting at or before this workgroup.
    // Every start is loaded before any is compared, so the loads issue
    // together (a test of b.count in the loop had split them into three
    // waits).
    uint32_t w[MAXB];
#pragma unroll
    for (int i = 1; i < MAXB; ++i) w[i] = b.wg_begin[i];
    int m = 0;
#pragma unroll
    for (int i = 1; i < MAXB; ++i) m += blockIdx.x >= w[i] ? 1 : 0;
    return m;
}

// The launch arguments of an N-pass workgroup's matrix, read in one round
// trip.  Read where each is used, the compiler had waited for each group of
// them in turn: 4-8 round trips of about 0.5 us before a pass streamed.
__device__ __forceinline__ MatArgs np_args(const BatchArgs& b, int mi) {
    MatArgs M = b.m[mi];
    asm volatile("" ::"s"(M.keys), "s"(M.n), "s"(M.wt), "s"(M.g), "s"(M.gw), "s"(M.gc), "s"(M.wsb), "s"(M.k),
                 "s"(M.max_iter), "s"(M.vec), "s"(M.fmt), "s"(M.kforce), "s"(M.wg_count), "s"(b.keep_frac),
                 "s"(b.out_half), "s"(b.inv_tau), "s"(b.wg_begin[mi]));
    return M;
}

// Stream a workgroup's share of a matrix.  Full rounds: the matrix is cut into
// tiles of U x GW x NP_THREADS weights that its workgroups take round-robin, so
// they sweep HBM together (measured: 10-20% faster than giving each workgroup
// one contiguous slice).  What is left after the last full round (under one
// tile per workgroup, plus the short last tile) is split evenly over the
// workgroups in steps of GW x NP_THREADS, so that no workgroup runs a whole
// extra tile after the others have finished.  In a tile a thread loads U groups
// of GW weights (ld), then computes all U results (cp: table lookups,
// atomics), then stores them (st); f1 handles single weights: the ragged tail,
// or everything when the buffers are not 16-byte aligned.
template <int U, int GW>
struct Slice {
    static constexpr uint64_t STEP = (uint64_t)GW * NP_THREADS;
    static constexpr uint64_t TILE = U * STEP;
    uint64_t nvec;     // weights in whole groups of GW
    uint64_t rounds;   // full rounds of tiles
    uint64_t rest0;    // first weight after the full rounds
    uint64_t per;      // steps of the rest per workgroup
    __device__ __forceinline__ explicit Slice(const MatArgs& M) {
        const uint64_t a = M.wg_count;
        nvec = M.n & ~(uint64_t)(GW - 1);
        rounds = nvec / TILE / a;
        rest0 = rounds * a * TILE;
        per = ((nvec - rest0 + STEP - 1) / STEP + a - 1) / a;
    }
    // weights one workgroup handles, at most (either path)
    __device__ __forceinline__ uint64_t bound(const MatArgs& M) const {
        const uint64_t scalar = (M.n + (uint64_t)M.wg_count * NP_THREADS - 1) /
                                ((uint64_t)M.wg_count * NP_THREADS) * NP_THREADS;
        return max(rounds * TILE + per * STEP, scalar) + NP_THREADS;
    }
};

// REV walks the same work in descending order (the rest first, then the rounds
// from the last), so that the grid sweeps the matrix from its end.  ld(i, c)
// loads with cached loads when c is std::true_type: for the tiles starting in
// [c_lo, c_hi), the part of the sweep that the next pass can find in the
// Infinity Cache; other tiles use non-temporal loads.
template <int U, int GW, bool REV = false, class Ld, class Cp, class St, class F1, class Full = std::nullptr_t>
__device__ __forceinline__ void for_slice(const MatArgs& M, uint32_t wl, uint64_t c_lo, uint64_t c_hi, Ld ld,
                                          Cp cp, St st, F1 f1, Full full = nullptr) {
    const uint64_t n = M.n;
    const uint64_t a = M.wg_count;
    if (!M.vec) {
        for (uint64_t j = (uint64_t)wl * NP_THREADS + threadIdx.x; j < n; j += a * NP_THREADS) f1(j);
        return;
    }
    using S = Slice<U, GW>;
    const S sh(M);
    using R = decltype(ld(0, std::true_type{}));
    using O = decltype(cp(R{}));
    auto round_c = [&](uint64_t b0, auto cached) {   // a full tile at b0
        const uint64_t i0 = b0 + (uint64_t)GW * threadIdx.x;
        R r[U];
#pragma unroll
        for (int u = 0; u < U; ++u) r[u] = ld(i0 + u * S::STEP, cached);
        __builtin_amdgcn_sched_barrier(0);   // all U loads issue before any use
        O o[U];
#pragma unroll
        for (int u = 0; u < U; ++u) o[u] = cp(r[u]);
#pragma unroll
        for (int u = 0; u < U; ++u) st(i0 + u * S::STEP, o[u]);
    };
    auto round = [&](uint64_t q) {         // this workgroup's full tile of round q
        const uint64_t b0 = ((uint64_t)wl + q * a) * S::TILE;
        if constexpr (!std::is_same_v<Full, std::nullptr_t>) {
            // the caller's own form of a full tile
            if (b0 >= c_lo && b0 < c_hi) full(b0, std::true_type{});
            else full(b0, std::false_type{});
        } else {
            if (b0 >= c_lo && b0 < c_hi) round_c(b0, std::true_type{});
            else round_c(b0, std::false_type{});
        }
    };
    auto rest_c = [&](uint64_t b0, uint64_t s1, auto cached) {
        const uint64_t i0 = b0 + (uint64_t)GW * threadIdx.x;
        R r[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i0 + u * S::STEP < s1) r[u] = ld(i0 + u * S::STEP, cached);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i0 + u * S::STEP < s1) st(i0 + u * S::STEP, cp(r[u]));
    };
    auto rest = [&]() {                    // this workgroup's steps of the rest
        const uint64_t s0 = sh.rest0 + (uint64_t)wl * sh.per * S::STEP;
        const uint64_t s1 = min(sh.nvec, s0 + sh.per * S::STEP);
        for (uint64_t b0 = s0; b0 < s1; b0 += S::TILE) {
            if (b0 >= c_lo && b0 < c_hi) rest_c(b0, s1, std::true_type{});
            else rest_c(b0, s1, std::false_type{});
        }
    };
    if (REV) {
        rest();
        for (uint64_t q = sh.rounds; q-- > 0;) round(q);
    } else {
        for (uint64_t q = 0; q < sh.rounds; ++q) round(q);
        rest();
    }
    if (wl == a - 1)
        for (uint64_t j = sh.nvec + threadIdx.x; j < n; j += NP_THREADS) f1(j);
}

// The cached part of a sweep over n weights: the last keep_frac of it, at the
// end (top) of the matrix for a forward sweep, at its start for REV.
__device__ __forceinline__ void cached_range(const BatchArgs& b, uint64_t n, bool rev, uint64_t& lo, uint64_t& hi) {
    const uint64_t k = (uint64_t)((double)n * (double)b.keep_frac);
    lo = rev ? 0 : n - k;
    hi = rev ? k : ~0ull;
}

struct Nothing {};

// Register images of one 8-weight group.
struct Keys8 { uint4 q; };
// ... and of one 4-weight group.
struct Keys4 { uint2 q; };
struct KeysG4 { uint2 q; float4 g; };
// ... with four 16-bit gradients, decoded only when used (after every load of
// the tile has issued).
struct KeysH4 { uint2 q; uint2 g; };
struct KeysH8 { uint4 q; uint4 g; };

// Paired key loads: a wave loads the keys of two 4-weight groups with one
// 16-byte load per lane (lanes 0-31 the first group's 256 keys, lanes 32-63
// the second's); lane l then takes its four keys of a group from lane
// src / 4 = l / 2 (first group) or 32 + l / 2 (second), the low or high half
// of that lane's 16 bytes as l is even or odd.  Every lane of the wave must
// take part (ds_bpermute).
__device__ __forceinline__ uint2 key_half(const uint4& kq, int src, bool odd) {
    auto bp = [&](uint32_t v) { return (uint32_t)__builtin_amdgcn_ds_bpermute(src, (int)v); };
    const uint32_t a0 = bp(kq.x), a1 = bp(kq.y), a2 = bp(kq.z), a3 = bp(kq.w);
    return odd ? make_uint2(a2, a3) : make_uint2(a0, a1);
}
__device__ __forceinline__ float4 g4_of(const KeysG4& r, int) { return r.g; }
__device__ __forceinline__ float4 g4_of(const KeysH4& r, int fmt) {
    return make_float4(grad_value(r.g.x & 0xFFFFu, fmt), grad_value(r.g.x >> 16, fmt),
                       grad_value(r.g.y & 0xFFFFu, fmt), grad_value(r.g.y >> 16, fmt));
}

typedef unsigned int v4u_t __attribute__((ext_vector_type(4)));
typedef unsigned int v2u_t __attribute__((ext_vector_type(2)));
typedef float v4f_t __attribute__((ext_vector_type(4)));
// Streaming loads and stores.  Consecutive N-sized passes sweep in opposite
// directions (histogram forward, W~ gather backward, keyed sum forward,
// gradient gather backward), so the last ~256 MB a pass reads with plain
// (cached) loads are still in the Infinity Cache where the next pass starts.
// Plain loads for the end of the key sweep in the histogram (for the W~
// gather), the W~ gather (for the keyed sum) and the keyed sum (for the
// gradient gather), as much as the cache holds (set_keep_frac); the rest is
// non-temporal (nt), which a pass runs a little faster with when nothing
// after it reads the same data.  The gathers' outputs use nt stores, float4
// or (16-bit W~) uint2: gradient gather 404 -> 381 us on the decoder layer,
// 16-bit W~ gather 168 -> 162 us, and the kernel after the W~ gather no
// longer inherits its dirty lines.
__device__ __forceinline__ uint4 ld_u4(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ uint2 ld_u2(const void* p) { return *reinterpret_cast<const uint2*>(p); }
__device__ __forceinline__ float4 ld_f4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ uint4 ld_u4_nt(const void* p) {
    const v4u_t v = __builtin_nontemporal_load(reinterpret_cast<const v4u_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 ld_u2_nt(const void* p) {
    const v2u_t v = __builtin_nontemporal_load(reinterpret_cast<const v2u_t*>(p));
    return make_uint2(v.x, v.y);
}
__device__ __forceinline__ float4 ld_f4_nt(const float* p) {
    const v4f_t v = __builtin_nontemporal_load(reinterpret_cast<const v4f_t*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st_f4_nt(float* p, float4 x) {
    __builtin_nontemporal_store(v4f_t{x.x, x.y, x.z, x.w}, reinterpret_cast<v4f_t*>(p));
}
__device__ __forceinline__ void st_u2_nt(void* p, uint2 x) {
    __builtin_nontemporal_store(v2u_t{x.x, x.y}, reinterpret_cast<v2u_t*>(p));
}
__device__ __forceinline__ void st_u4_nt(void* p, uint4 x) {
    __builtin_nontemporal_store(v4u_t{x.x, x.y, x.z, x.w}, reinterpret_cast<v4u_t*>(p));
}

// ----------------------------------------------------------------------------
// init_unique: zero, histogram, partial merge, window selection

__global__ void __launch_bounds__(T_THREADS) k_init_zero(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    const MatArgs& M = b.m[blockIdx.y];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    for (int u = blockIdx.x * T_THREADS + threadIdx.x; u < NKEYS; u += gridDim.x * T_THREADS)
        ws.counts[u] = 0u;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        DevState* st = ws.st;
        st->teff = 0;
        st->conv = 0;
        st->nonfinite = 0u;
        st->num_unique = 0u;
    }
}

// Pattern histogram.  Magnitudes [0, W4) of both signs (|w| < 16) count in
// LDS; anything else goes straight to the global counts with an atomic.
// Each workgroup then writes the occupied span of its LDS histogram as packed
// 16-bit counts (two bins per word); a bin that reached 2^16 in this
// workgroup is added to the global counts instead.
__global__ void __launch_bounds__(NP_THREADS) k_hist(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ __align__(16) uint32_t h[2 * W4];
    __shared__ int red[2];
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    for (int i = threadIdx.x; i < 2 * W4 / 4; i += NP_THREADS) reinterpret_cast<uint4*>(h)[i] = uint4{0u, 0u, 0u, 0u};
    if (threadIdx.x == 0) { red[0] = W4; red[1] = 0; }
    __syncthreads();
    const uint16_t* keys = M.keys;
    uint32_t* gcounts = ws.counts;
    auto add = [&](uint32_t key) {
        const uint32_t mag = key & 0x7FFFu;
        if (mag < (uint32_t)W4) atomicAdd(&h[(key >> 15) * W4 + mag], 1u);
        else atomicAdd(&gcounts[key], 1u);
    };
    // Cached loads at the end of this forward sweep: it stays in the Infinity
    // Cache, where the W~ gather, sweeping backwards, starts.
    uint64_t c_lo, c_hi;
    cached_range(b, M.n, false, c_lo, c_hi);
    for_slice<4, 8>(M, wl, c_lo, c_hi,
        [&](uint64_t i, auto c) { return Keys8{c ? ld_u4(keys + i) : ld_u4_nt(keys + i)}; },
        [&](const Keys8& r) {
            add(r.q.x & 0xFFFFu); add(r.q.x >> 16);
            add(r.q.y & 0xFFFFu); add(r.q.y >> 16);
            add(r.q.z & 0xFFFFu); add(r.q.z >> 16);
            add(r.q.w & 0xFFFFu); add(r.q.w >> 16);
            return Nothing{};
        },
        [&](uint64_t, Nothing) {},
        [&](uint64_t i) { add(keys[i]); });
    __syncthreads();
    EDKM_STAMP_MARK(b, 2);   // keys streamed
    // occupied span [lo, hi) over both signs, rounded out to even magnitudes;
    // a thread's W4 / NP_THREADS magnitudes are read all at once (as a loop
    // each read waited for the previous one)
    int lo = W4, hi = 0;
    {
        constexpr int PER = W4 / NP_THREADS;
        uint32_t x[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) x[q] = h[threadIdx.x + q * NP_THREADS] | h[W4 + threadIdx.x + q * NP_THREADS];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int mag = threadIdx.x + q * NP_THREADS;
            if (x[q]) { lo = min(lo, mag); hi = max(hi, mag + 1); }
        }
    }
    lo = wave_reduce(lo, 0x7FFFFFFF, op_min);   // one LDS atomic per wave
    hi = wave_reduce(hi, -0x7FFFFFFF - 1, op_max);
    if ((threadIdx.x & 63) == 0) {
        atomicMin(&red[0], lo);
        atomicMax(&red[1], hi);
    }
    __syncthreads();
    EDKM_STAMP_MARK(b, 3);   // span found
    lo = red[0] & ~1;
    hi = (red[1] + 1) & ~1;
    if (hi <= lo) { lo = 0; hi = 0; }
    const int half = (hi - lo) >> 1;
    uint32_t* row = ws.part + (size_t)wl * ROW4;
    // four of a thread's pairs per round, every LDS read issued before the
    // first is used
    constexpr int RU = 4;
    for (int p0 = threadIdx.x; p0 < 2 * half; p0 += RU * NP_THREADS) {
        uint32_t c[RU][2];
#pragma unroll
        for (int q = 0; q < RU; ++q) {
            const int p = p0 + q * NP_THREADS;
            const int s = p >= half;
            const int mag = lo + 2 * (p - s * half);
            if (p < 2 * half) { c[q][0] = h[s * W4 + mag]; c[q][1] = h[s * W4 + mag + 1]; }
        }
#pragma unroll
        for (int q = 0; q < RU; ++q) {
            const int p = p0 + q * NP_THREADS;
            if (p >= 2 * half) break;
            const int s = p >= half;
            const int mag = lo + 2 * (p - s * half);
            uint32_t c0 = c[q][0], c1 = c[q][1];
            if (c0 > 0xFFFFu) { atomicAdd(&gcounts[(s << 15) | mag], c0); c0 = 0u; }
            if (c1 > 0xFFFFu) { atomicAdd(&gcounts[(s << 15) | (mag + 1)], c1); c1 = 0u; }
            __builtin_nontemporal_store(c0 | (c1 << 16), row + p);   // read once, by the merge
        }
    }
    if (threadIdx.x == 0) ws.span[wl] = make_int2(lo, hi);
}

// Partial-row merges.  Thread = one bin (or bin pair), blockIdx.y = a chunk of
// MERGE_ROWS rows, blockIdx.z = matrix; each thread sums its chunk with
// independent accumulators and adds the chunk total to the destination with
// one atomic, so a matrix's merge is spread over many threads instead of
// walking all of its rows in one.
constexpr int MERGE_ROWS = 16;
constexpr int MERGE_THREADS = 256;

// Histogram rows (packed 16-bit pairs over per-row spans) into counts.
// Grid (W4 / MERGE_THREADS, row chunks, count).
__global__ void __launch_bounds__(MERGE_THREADS) k_hist_merge(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    const MatArgs& M = b.m[blockIdx.z];
    const int wg_count = (int)M.wg_count;
    asm volatile("" ::"s"(wg_count), "s"(M.wsb), "s"(M.max_iter));   // the arguments, in one wait
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int r0 = blockIdx.y * MERGE_ROWS;
    const int r1 = min(wg_count, r0 + MERGE_ROWS);
    if (r0 >= r1) return;
    const int q = blockIdx.x * MERGE_THREADS + threadIdx.x;   // < W4 pairs
    const int s = q >= W4 / 2;
    const int mag = 2 * (q - s * (W4 / 2));
    uint32_t s0 = 0u, s1 = 0u;
    const uint32_t* part = ws.part;
    // Every row's span first, then every row's word, all in flight at once.
    // (Loaded under the row test, each span load -- a scalar load -- had
    // waited for the previous one: 16 round trips, 8 us per block.)
    int2 lh[MERGE_ROWS];
#pragma unroll
    for (int q2 = 0; q2 < MERGE_ROWS; ++q2) lh[q2] = ws.span[min(r0 + q2, r1 - 1)];
    uint32_t x[MERGE_ROWS];
#pragma unroll
    for (int q2 = 0; q2 < MERGE_ROWS; ++q2) {
        const int r = r0 + q2;
        x[q2] = 0u;
        if (r < r1 && mag >= lh[q2].x && mag < lh[q2].y)
            x[q2] = part[(size_t)r * ROW4 + s * ((lh[q2].y - lh[q2].x) >> 1) + ((mag - lh[q2].x) >> 1)];
    }
#pragma unroll
    for (int q2 = 0; q2 < MERGE_ROWS; ++q2) {
        s0 += x[q2] & 0xFFFFu;
        s1 += x[q2] >> 16;
    }
    EDKM_STAMP_MARK(b, 2);   // rows summed
    uint32_t* c = ws.counts + (s << 15) + mag;
    if (s0) atomicAdd(c, s0);
    if (s1) atomicAdd(c + 1, s1);
}

// Window selection: one block per matrix, grid (1, count).  Wave w owns the
// SPAN = 2048 magnitudes [2048 w, 2048 w + 2048) of both signs, in NCH = 8
// chunks of 256; lane l holds the 4 consecutive magnitudes 4 l .. 4 l + 3 of
// each chunk, so that loads and LDS stores are contiguous across the wave.  The
// block builds in LDS the running count of weights over finite magnitudes
// (within each wave's span, plus a per-wave offset) and reduces the
// occupied-pattern count, the non-finite flag, the occupied finite magnitude
// range and the sum of squared counts (for the keyed-sum mode).  A window of
// width W covers the whole occupied range when it fits, else the W consecutive
// magnitudes holding the most weights (lowest start on ties).
__global__ void __launch_bounds__(NP_THREADS) k_window(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    constexpr int NW = NP_THREADS / 64;
    constexpr int SPAN = MAGS / NW;
    constexpr int NCH = SPAN / 256;
    __shared__ __align__(16) uint32_t pre[MAGS];   // weights with finite magnitude in [2048 w, x], w = x / 2048
    __shared__ uint32_t woff[NW + 1];     // weights with finite magnitude < 2048 w
    __shared__ int wred[4][NW];           // per wave: lo, hi, occupied patterns, non-finite
    __shared__ unsigned long long wsq[NW];
    __shared__ int red[4];                // the block's: lo, hi, occupied patterns, non-finite
    __shared__ unsigned long long sqsum, best[2];
    const MatArgs& M = b.m[blockIdx.y];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int fin = fin_mags(M.fmt);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int mw = wave * SPAN + 4 * lane;   // this lane's first magnitude; chunk j adds 256 j
    // best[] is first used after two barriers below
    if (threadIdx.x == 0) { best[0] = 0ull; best[1] = 0ull; }
    uint4 p[NCH], q[NCH];
    {
        const uint4* p4 = reinterpret_cast<const uint4*>(ws.counts + mw);
        const uint4* q4 = reinterpret_cast<const uint4*>(ws.counts + MAGS + mw);
#pragma unroll
        for (int j = 0; j < NCH; ++j) { p[j] = p4[64 * j]; q[j] = q4[64 * j]; }
    }
    // bit 4 j + e of the masks: magnitude mw + 256 j + e (ascending with the bit)
    uint32_t occp = 0u, occn = 0u, finm = 0u, carry = 0u;
    unsigned long long sq = 0ull;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const bool f = mw + 256 * j < fin;     // the finite ranges end on a multiple of 4
        const uint32_t a[4] = {p[j].x, p[j].y, p[j].z, p[j].w};
        const uint32_t c[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
        uint32_t s4[4], run = 0u;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            occp |= (uint32_t)(a[e] != 0u) << (4 * j + e);
            occn |= (uint32_t)(c[e] != 0u) << (4 * j + e);
            const uint32_t ae = f ? a[e] : 0u, ce = f ? c[e] : 0u;
            sq += (unsigned long long)ae * ae;
            sq += (unsigned long long)ce * ce;
            run += ae + ce;
            s4[e] = run;
        }
        finm |= (f ? 0xFu : 0u) << (4 * j);
        const uint32_t x = wave_incl_scan(run);   // over the wave's lanes
        const uint32_t base = carry + x - run;
        *reinterpret_cast<uint4*>(pre + mw + 256 * j) =
            make_uint4(base + s4[0], base + s4[1], base + s4[2], base + s4[3]);
        carry += (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
    }
    EDKM_STAMP_MARK(b, 2);   // wave 0's share of the counts scanned
    const uint32_t occ = (occp | occn) & finm;
    auto bit_mag = [&](int bit) { return mw + 256 * (bit >> 2) + (bit & 3); };
    int lo = occ ? bit_mag(__builtin_ctz(occ)) : 1 << 30;
    int hi = occ ? bit_mag(31 - __builtin_clz(occ)) : -1;
    int nu = __builtin_popcount(occp) + __builtin_popcount(occn);
    int nf = ((occp | occn) & ~finm) != 0u;
    lo = wave_reduce(lo, 0x7FFFFFFF, op_min);
    hi = wave_reduce(hi, -0x7FFFFFFF - 1, op_max);
    nu = wave_reduce(nu, 0, op_add);
    nf = wave_reduce(nf, 0, op_or);
    sq = wave_sum_u64(sq);
    // each wave's results go to slots of its own; wave 0 combines them after
    // the barrier (no LDS word is written by two waves)
    if (lane == 0) {
        woff[wave + 1] = carry;
        wred[0][wave] = lo;
        wred[1][wave] = hi;
        wred[2][wave] = nu;
        wred[3][wave] = nf;
        wsq[wave] = sq;
    }
    __syncthreads();
    if (wave == 0) {
        // wave 0 combines the NW slots, lane w taking wave w's (a serial loop
        // over them in one thread, each step waiting on the previous LDS
        // write, had taken 4 of this kernel's 7.5 us)
        const bool in = lane < NW;
        const uint32_t x = wave_incl_scan(in ? woff[lane + 1] : 0u);
        const int r0 = wave_reduce(in ? wred[0][lane] : 0x7FFFFFFF, 0x7FFFFFFF, op_min);
        const int r1 = wave_reduce(in ? wred[1][lane] : -0x7FFFFFFF - 1, -0x7FFFFFFF - 1, op_max);
        const int r2 = wave_reduce(in ? wred[2][lane] : 0, 0, op_add);
        const int r3 = wave_reduce(in ? wred[3][lane] : 0, 0, op_or);
        const unsigned long long q = wave_sum_u64(in ? wsq[lane] : 0ull);
        if (in) woff[lane + 1] = x;
        if (lane == 0) {
            woff[0] = 0u;
            red[0] = r0; red[1] = r1; red[2] = r2; red[3] = r3;
            sqsum = q;
        }
    }
    __syncthreads();
    EDKM_STAMP_MARK(b, 3);   // block totals combined
    const int mlo = red[0], mhi = red[1];
    auto P = [&](int x) -> uint32_t {   // weights with finite magnitude < x
        return x == 0 ? 0u : pre[x - 1] + woff[(x - 1) / SPAN];
    };
    int wl[2], ww[2];
    const int widths[2] = {W4, W8};
#pragma unroll
    for (int w = 0; w < 2; ++w) {
        const int W = widths[w];
        if (mhi < 0) { wl[w] = 0; ww[w] = 0; continue; }
        if (mhi - mlo + 1 <= W) { wl[w] = mlo; ww[w] = mhi - mlo + 1; continue; }
        unsigned long long mine = 0ull;
        for (int s = mlo + threadIdx.x; s <= mhi - W + 1; s += NP_THREADS) {
            const uint32_t cov = P(s + W) - P(s);
            // larger coverage wins, then the smaller start
            const unsigned long long key = ((unsigned long long)cov << 32) | (uint32_t)(0x7FFFFFFF - s);
            mine = key > mine ? key : mine;
        }
        mine = wave_max_u64(mine);   // one LDS atomic per wave, not per thread
        if ((threadIdx.x & 63) == 0) atomicMax(&best[w], mine);
        __syncthreads();
        wl[w] = 0x7FFFFFFF - (int)(uint32_t)(best[w] & 0xFFFFFFFFull);
        ww[w] = W;
    }
    if (threadIdx.x == 0) {
        EDKM_STAMP_MARK(b, 4);   // windows chosen
        const uint32_t total = woff[NW];
        // expected number of other lanes sharing an address in a 64-lane keyed atomic
        const double e = total ? 2016.0 * (double)sqsum / ((double)total * (double)total) : 0.0;
        DevState* st = ws.st;
        st->num_unique = (uint32_t)red[2];
        st->nonfinite = (uint32_t)red[3];
        st->mlo = mlo;
        st->mhi = mhi;
        st->lo4 = wl[0]; st->w4 = ww[0];
        st->lo8 = wl[1]; st->w8 = ww[1];
        st->kmode = M.kforce >= 0 ? M.kforce : (e > KEYED_U64_ABOVE ? KEYED_U64 : KEYED_I32);
        if (M.nuniq_out) *M.nuniq_out = (uint32_t)red[2];
    }
}

// ----------------------------------------------------------------------------
// forward table phase

// Table keys of a thread: T_KPT per thread over T_WG blocks x T_THREADS threads
// (= 65,536).  Kernels load everything the 4 patterns need first and compute
// afterwards, so the loads overlap instead of forming a chain.
__device__ __forceinline__ int table_key(int r) {
    return blockIdx.x * T_THREADS + threadIdx.x + r * (T_WG * T_THREADS);
}

// Iteration t (1..max_iter): C^(t-1) from the partials of iteration t-1 (or
// c_in), early stop test, then this block's partial S_j = sum n_u a_uj and
// P_j = sum n_u a_uj v_u.  Grid (T_WG, count).
template <int K>
__global__ void __launch_bounds__(T_THREADS) k_fwd_iter(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float red[BLOCK_TOTAL_LDS(2 * K)];
    __shared__ float csh[K];
    __shared__ int stop;
    const MatArgs& M = b.m[blockIdx.y];
    const int t = b.t;
    // Every load first, with no branch in between (a branch or an early
    // return between them had the compiler wait for each scalar load before
    // issuing the next, 2-3 round trips): the pattern counts, the previous
    // iteration's partial block and C^(t-2) (at t = 1: c_in, and partial row 0,
    // unused), the convergence flag.  Indices are clamped for launches past
    // this matrix's max_iter, which return below.
    const float* c_in = M.c_in;
    const int max_iter = M.max_iter, fmt = M.fmt;
    const float eps = b.eps, s2 = b.s2;
    // the arguments, in one wait
    asm volatile("" ::"s"(c_in), "s"(max_iter), "s"(fmt), "s"(t), "s"(eps), "s"(s2), "s"(M.wsb));
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int tl = max(1, min(t, max_iter));
    uint32_t n4[T_KPT];
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) n4[r] = ws.counts[table_key(r)];
    PartCols<2 * K> pc;
    pc.load_block(ws.tpart + (size_t)(tl - 1) * T_WG * PSTRIDE);
    const float* cp = tl > 1 ? ws.chist + (tl - 2) * KMAX : c_in;
    const float cprev = cp[threadIdx.x % K];
    DevState* st = ws.st;
    const int conv = st->conv;
    EDKM_STAMP_MARK(b, 2);   // loads issued
    if (t > max_iter) return;
    const bool lead = blockIdx.x == 0;
    if (t == 1) {
        if (threadIdx.x < K) {
            csh[threadIdx.x] = cprev;
            if (lead) { ws.chist[threadIdx.x] = cprev; ws.shist[threadIdx.x] = 0.f; }
        }
        if (lead && threadIdx.x == 0) { st->conv = 0; st->teff = 0; }
        __syncthreads();
    } else {
        if (threadIdx.x == 0) stop = 0;
        pc.stage(red);
        if (conv) return;
        if (threadIdx.x < K) {
            const int j = threadIdx.x;
            const float S = PartCols<2 * K>::total(red, j), P = PartCols<2 * K>::total(red, K + j);
            const float cn = S > 0.f ? P / S : cprev;
            csh[j] = cn;
            if (lead) { ws.chist[(t - 1) * KMAX + j] = cn; ws.shist[(t - 1) * KMAX + j] = S; }
            if (eps > 0.f && !(fabsf(cn - cprev) <= eps)) atomicOr(&stop, 1);
        }
        __syncthreads();
        if (eps > 0.f && stop == 0) {   // max_j |C^(t-1) - C^(t-2)| <= eps: T = t - 1
            if (lead && threadIdx.x == 0) { st->teff = t - 1; st->conv = 1; }
            return;
        }
    }
    EDKM_STAMP_MARK(b, 3);   // partial block summed, C formed
    float c[K];
#pragma unroll
    for (int j = 0; j < K; ++j) c[j] = csh[j];
    float acc[2 * K];
#pragma unroll
    for (int j = 0; j < 2 * K; ++j) acc[j] = 0.f;
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) {
        const int u = table_key(r);
        const uint32_t n = n4[r];
        if (n == 0u || !key_finite(u, fmt)) continue;
        const float v = key_value(u, fmt);
        float a[K];
        attn_row<K>(v, c, s2, a);
        const float nf = (float)n;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const float w = nf * a[j];
            acc[j] += w;
            acc[K + j] = fmaf(w, v, acc[K + j]);
        }
    }
    EDKM_STAMP_MARK(b, 4);   // patterns done
    const float tot = block_total<2 * K>(acc, red);
    EDKM_STAMP_MARK(b, 5);   // block summed
    if (threadIdx.x < 2 * K) ws.tpart[((size_t)t * T_WG + blockIdx.x) * PSTRIDE + threadIdx.x] = tot;
}

// After the last iteration: C^(T), c_out, T; per occupied pattern the W~ value
// Tab_u = sum_j a^(T)_uj C^(T)_j (a^(T) built from C^(T-1)) and
// H_u = -(1/tau) sum_j a^(T)_uj (C^(T)_j - Tab_u) sgn(v_u - C^(T-1)_j);
// clears G.  Grid (T_WG, count).
template <int K>
__global__ void __launch_bounds__(T_THREADS) k_fwd_out(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float red[T_THREADS];
    __shared__ float cT[K], cP[K];
    const MatArgs& M = b.m[blockIdx.y];
    // the arguments, in one wait (read where they are used, each had cost a
    // round trip of its own)
    const int max_iter = M.max_iter, fmt = M.fmt;
    float* const c_out = M.c_out;
    int32_t* const iters_out = M.iters_out;
    const float s2 = b.s2, inv_tau = b.inv_tau;
    asm volatile("" ::"s"(max_iter), "s"(fmt), "s"(c_out), "s"(iters_out), "s"(s2), "s"(inv_tau), "s"(M.wsb));
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    // every load first (the partial block and C^(T-1) of a run that did all
    // max_iter iterations, the convergence state; an early stop reads its two
    // rows afterwards)
    DevState* st = ws.st;
    const int conv = st->conv, teff = st->teff;
    uint32_t n4[T_KPT];
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) n4[r] = ws.counts[table_key(r)];
    PartCols<2 * K> pc;
    pc.load_block(ws.tpart + (size_t)max_iter * T_WG * PSTRIDE);
    const float cprev = ws.chist[(max_iter - 1) * KMAX + threadIdx.x % K];
    const bool lead = blockIdx.x == 0;
    pc.stage(red);
    int T;
    if (conv) {
        T = teff;
        if (threadIdx.x < K) {
            cT[threadIdx.x] = ws.chist[T * KMAX + threadIdx.x];
            cP[threadIdx.x] = ws.chist[(T - 1) * KMAX + threadIdx.x];
        }
        __syncthreads();
    } else {
        T = max_iter;
        if (threadIdx.x < K) {
            const int j = threadIdx.x;
            const float S = PartCols<2 * K>::total(red, j), P = PartCols<2 * K>::total(red, K + j);
            const float cn = S > 0.f ? P / S : cprev;
            cT[j] = cn;
            cP[j] = cprev;
            if (lead) { ws.chist[T * KMAX + j] = cn; ws.shist[T * KMAX + j] = S; }
        }
        if (lead && threadIdx.x == 0) st->teff = T;
        __syncthreads();
    }
    if (lead) {
        if (threadIdx.x < K) {
            c_out[threadIdx.x] = cT[threadIdx.x];
            ws.cfin[threadIdx.x] = cP[threadIdx.x];          // for k_grad_top, which does not know T
            ws.cfin[KMAX + threadIdx.x] = cT[threadIdx.x];
        }
        if (threadIdx.x == 0 && iters_out) *iters_out = T;
    }
    float c1[K], c0[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c1[j] = cT[j]; c0[j] = cP[j]; }
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) {
        const int u = table_key(r);
        ws.G[u] = 0.f;
        const uint32_t n = n4[r];
        if (n == 0u) continue;
        if (!key_finite(u, fmt)) { ws.tab[u] = __builtin_nanf(""); ws.H[u] = __builtin_nanf(""); continue; }
        const float v = key_value(u, fmt);
        float a[K], d[K], c1m;
        attn_row_sel<K>(v, c0, s2, a, c1, c1m);
        const float tv = centroid_dev<K>(a, c1, c1m, d);
        float h = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) h = fmaf(a[j] * d[j], sgnf(v - c0[j]), h);
        ws.tab[u] = tv;
        ws.H[u] = -h * inv_tau;
    }
}

// ----------------------------------------------------------------------------
// N-sized gathers and the keyed reduction

// W~_i = Tab[bits_i]; the window [lo4, lo4 + w4) of the table sits in LDS.
__global__ void __launch_bounds__(NP_THREADS) k_gather_wt(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float tw[2 * W4];
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    const int lo = ws.st->lo4, w = ws.st->w4;
    const float* tab = ws.tab;
    fill_lds<2 * W4, NP_THREADS>(tw, tab, 2 * w, [&](int i) {
        const int s = i >= w;
        return (s << 15) | (lo + i - s * w);
    });
    __syncthreads();
    // Lookup, written as an LDS read at a clamped index that lanes outside the
    // window overwrite with a global read: the compiler turns this into a
    // per-lane address select and one flat load, with no branch.  The plain
    // two-way conditional compiled to a branch per lookup (3% slower in the
    // gradient gather); a true LDS read plus a separately predicated global
    // read was 7% slower.
    auto look = [&](uint32_t key) -> float {
        const uint32_t d = (key & 0x7FFFu) - (uint32_t)lo;
        const bool in = d < (uint32_t)w;
        float v = tw[(key >> 15) * w + (in ? d : 0u)];
        if (!in) v = tab[key];
        return v;
    };
    auto look4 = [&](uint32_t k0, uint32_t k1, uint32_t k2, uint32_t k3) {
        return make_float4(look(k0), look(k1), look(k2), look(k3));
    };
    const uint16_t* keys = M.keys;
    uint64_t c_lo, c_hi;
    cached_range(b, M.n, true, c_lo, c_hi);
    if (b.out_half) {
        uint16_t* out = reinterpret_cast<uint16_t*>(M.wt);
        auto h2 = [&](float a, float c) -> uint32_t {
            return to_half_bits(a, M.fmt) | (to_half_bits(c, M.fmt) << 16);
        };
        // 16-byte key loads and stores, 8 weights per lane and group (with
        // 8-byte ones, 4 weights, this path ran at 5.3 instead of 5.6 TB/s)
        for_slice<8, 8, true>(M, wl, c_lo, c_hi,
            [&](uint64_t i, auto c) { return Keys8{c ? ld_u4(keys + i) : ld_u4_nt(keys + i)}; },
            [&](const Keys8& r) {
                const float4 v = look4(r.q.x & 0xFFFFu, r.q.x >> 16, r.q.y & 0xFFFFu, r.q.y >> 16);
                const float4 u = look4(r.q.z & 0xFFFFu, r.q.z >> 16, r.q.w & 0xFFFFu, r.q.w >> 16);
                return make_uint4(h2(v.x, v.y), h2(v.z, v.w), h2(u.x, u.y), h2(u.z, u.w));
            },
            [&](uint64_t i, uint4 o) { st_u4_nt(out + i, o); },
            [&](uint64_t i) { out[i] = (uint16_t)to_half_bits(look(keys[i]), M.fmt); });
    } else {
        float* out = reinterpret_cast<float*>(M.wt);
        // (paired 16-byte key loads, as in the gradient gather, made this pass
        // 1-2% slower: 198 -> 201 us on the decoder layer)
        for_slice<16, 4, true>(M, wl, c_lo, c_hi,
            [&](uint64_t i, auto c) { return Keys4{c ? ld_u2(keys + i) : ld_u2_nt(keys + i)}; },
            [&](const Keys4& r) {
                return look4(r.q.x & 0xFFFFu, r.q.x >> 16, r.q.y & 0xFFFFu, r.q.y >> 16);
            },
            [&](uint64_t i, float4 o) { st_f4_nt(out + i, o); },
            [&](uint64_t i) { out[i] = look(keys[i]); });
    }
}

// G_u = sum over weights with pattern u of dL/dW~_i.
//
// LDS fp32 atomics run at a fraction of the integer rate on this GPU, so the
// window sums are kept in fixed point, q = round(g 2^S), added with integer LDS
// atomics.  Each workgroup chooses S from a first sample of its own g (one
// value per thread).  Values above the sample-based limit (and Inf/NaN) are
// added in fp32 to the global G, as are patterns outside the window.  G enters
// the backward only through the k-vector sums gamma and E over all patterns,
// where the fixed-point resolution is far below fp32 rounding.  Each workgroup
// ends by writing its window as one fp32 partial row.  Two accumulator modes,
// chosen per matrix by k_window from how concentrated the patterns are:
//
// KEYED_I32: 32-bit sums over the 4-byte window, added with atomics that
// return the previous value.  Every value with exponent <= L quantises below
// 2^30, where L is the sample's largest exponent, or its mean exponent + 8 if
// that is smaller, plus 2 (resolution at least 2^-19 of a value of mean
// exponent; a few huge values in the sample cannot coarsen the bulk).  A sum
// that wraps past the 32-bit range is detected from the returned value and the
// wrap (exactly +-2^32 quanta) goes to G in fp32, so no sum is ever lost.
//
// KEYED_U64: 64-bit sums over the 8-byte window with plain atomics.  Every
// value with exponent <= E + 6 (E the sample maximum) stays below 2^(61 - b)
// for a slice of at most 2^b weights, so no sum can overflow; the resolution
// is 2^(b - 55) of the sample maximum.
//
// Returning atomics serialise lanes that hit the same address, plain ones do
// not: with fp16 weights (about 0.23 other lanes per 64-lane atomic share an
// address) the 32-bit mode is 10% faster, with bf16 weights (about 1.8) the
// 64-bit mode is 30% faster.
constexpr int KW16_U = 8, KI16_U = 6;   // keyed sum with 16-bit dL/dW~: 64-bit, 32-bit mode
constexpr int GG16_U = 6;               // gradient gather with 16-bit dL/dW~ and dL/dw (8-weight groups)
template <bool G16>
__global__ void __launch_bounds__(NP_THREADS) k_keyed_grad(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ __align__(16) unsigned long long lds[2 * W8];   // 64-bit sums, or the 32-bit ones
    __shared__ int emax_sh, esum_sh, ecnt_sh;
    static_assert(2 * W4 * sizeof(int) <= sizeof(lds), "32-bit window fits the LDS buffer");
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    const DevState* st = ws.st;
    const bool wide = st->kmode == KEYED_U64;
    const int lo = wide ? st->lo8 : st->lo4, w = wide ? st->w8 : st->w4;
    const uint16_t* keys = M.keys;
    const float* g = M.g;
    const uint16_t* gh = reinterpret_cast<const uint16_t*>(M.g);   // G16: 16-bit patterns
    const int fmt = M.fmt;
    auto g1 = [&](uint64_t i) { return G16 ? grad_value(gh[i], fmt) : g[i]; };
    auto ldkg = [&](uint64_t i, auto c) {
        const uint2 k = c ? ld_u2(keys + i) : ld_u2_nt(keys + i);
        if constexpr (G16) return KeysH4{k, ld_u2_nt(gh + i)};
        else return KeysG4{k, ld_f4_nt(g + i)};
    };
    // tile depths (loads in flight per thread): 16-bit gradients move fewer
    // bytes per load, so they take deeper tiles
    constexpr int KW_U = G16 ? KW16_U : 4, KI_U = G16 ? KI16_U : 3;
    int* acc32 = reinterpret_cast<int*>(lds);
    {   // 16-byte LDS writes over the window (2 w words of 4 or 8 bytes), rounded up
        const int n16 = wide ? w : (2 * w + 3) / 4;
        for (int i = threadIdx.x; i < n16; i += NP_THREADS) reinterpret_cast<uint4*>(lds)[i] = uint4{0u, 0u, 0u, 0u};
    }
    if (threadIdx.x == 0) { emax_sh = 0; esum_sh = 0; ecnt_sh = 0; }
    // Clear the backward's first partial block, which k_grad_top adds into
    // next; the previous backward's reads of it are over.
    for (uint32_t i = wl * NP_THREADS + threadIdx.x; i < (uint32_t)(T_WG * PSTRIDE); i += M.wg_count * NP_THREADS)
        ws.bpart[i] = 0.f;
    __syncthreads();
    {   // sample: 64 consecutive values per wave, the waves' runs spread over the
        // matrix (one value per thread at scattered indices had cost a 128-byte
        // line per value, 33 MB per decoder layer); exponents of the normal
        // finite values: largest, sum and count
        const uint64_t runs = M.n > 64 ? M.n - 63 : 1;
        const uint64_t run0 = (((uint64_t)wl * (NP_THREADS / 64) + (threadIdx.x >> 6)) * 2654435761ull) % runs;
        const uint64_t i = min(run0 + (threadIdx.x & 63), M.n - 1);
        const int e = (int)((__float_as_uint(g1(i)) >> 23) & 0xFFu);
        const bool use = e != 0 && e != 0xFF;
        int smax = use ? e : 0, ssum = smax, scnt = use ? 1 : 0;
        smax = wave_reduce(smax, 0, op_max);
        ssum = wave_reduce(ssum, 0, op_add);
        scnt = wave_reduce(scnt, 0, op_add);
        if ((threadIdx.x & 63) == 0) {
            atomicMax(&emax_sh, smax);
            atomicAdd(&esum_sh, ssum);
            atomicAdd(&ecnt_sh, scnt);
        }
    }
    __syncthreads();
    float* G = ws.G;
    uint64_t c_lo, c_hi;
    cached_range(b, M.n, false, c_lo, c_hi);
    // The end of the key sweep cached, g non-temporal: those keys stay in the
    // Infinity Cache for the gradient gather, which sweeps backwards.
    auto stream = [&](auto add) {
        for_slice<KW_U, 4>(M, wl, c_lo, c_hi, ldkg,
            [&](const auto& r) {
                const float4 gv = g4_of(r, fmt);
                add(r.q.x & 0xFFFFu, gv.x); add(r.q.x >> 16, gv.y);
                add(r.q.y & 0xFFFFu, gv.z); add(r.q.y >> 16, gv.w);
                return Nothing{};
            },
            [&](uint64_t, Nothing) {},
            [&](uint64_t i) { add(keys[i], g1(i)); });
    };
    float* row = reinterpret_cast<float*>(ws.part) + (size_t)wl * ROW4;
    if (wide) {
        const int bn = 64 - __clzll((unsigned long long)Slice<KW_U, 4>(M).bound(M) - 1);   // 2^bn >= weights added here
        const int emax = emax_sh;
        const int S = 181 - bn - emax;               // 2^(emax-126) * 2^S = 2^(55-bn)
        const uint32_t elim = (uint32_t)min(emax + 6, 0xFE);
        stream([&](uint32_t key, float gv) {
            const uint32_t d = (key & 0x7FFFu) - (uint32_t)lo;
            const uint32_t e = (__float_as_uint(gv) >> 23) & 0xFFu;
            if (d < (uint32_t)w && e <= elim) {
                const long long q = __float2ll_rn(ldexpf(gv, S));
                atomicAdd(&lds[(key >> 15) * w + d], (unsigned long long)q);
            } else {
                atomicAdd(&G[key], gv);
            }
        });
        __syncthreads();
        for (int i = threadIdx.x; i < 2 * w; i += NP_THREADS)
            __builtin_nontemporal_store((float)ldexp((double)(long long)lds[i], -S), row + i);
    } else {
        // Values with exponent <= elim go to LDS: the sample maximum, but at most
        // 2^10 above the mean exponent.  Capped so the wrap value 2^(32 - S)
        // stays finite.
        const int emean = ecnt_sh > 0 ? (esum_sh + ecnt_sh / 2) / ecnt_sh : 0;
        const int elim = min(min(emax_sh, emean + 8) + 2, 190);
        const int S = 156 - elim;                    // |g 2^S| < 2^30
        const float wrap = ldexpf(1.0f, 32 - S);     // one turn of the 32-bit accumulator, as a value
        // One weight: its LDS atomic (returning the previous value), plus the
        // global add when it is not taken in LDS.  Every lane issues the LDS
        // atomic, the others adding 0 to a spare word of their own past the
        // window (one per lane: a shared one would be a uniform address, which
        // the compiler turns back into a branch): no branch then writes the
        // registers a pending return targets, and the wrap test (separate)
        // lets a whole tile's atomics issue before the first return is awaited.
        auto issue = [&](uint32_t key, float gv, int& q, int& old) {
            const uint32_t d = (key & 0x7FFFu) - (uint32_t)lo;
            const int e = (int)((__float_as_uint(gv) >> 23) & 0xFFu);
            const bool in = d < (uint32_t)w && e <= elim;
            q = in ? __float2int_rn(ldexpf(gv, S)) : 0;
            old = atomicAdd(&acc32[in ? (key >> 15) * w + d : 2 * W4 + (threadIdx.x & 63)], q);
            if (!in) atomicAdd(&G[key], gv);
        };
        auto settle = [&](uint32_t key, int q, int old) {   // (q, old) = (0, 0) never wraps
            const int sum = (int)((uint32_t)old + (uint32_t)q);
            if (((old ^ sum) & (q ^ sum)) < 0) atomicAdd(&G[key], q > 0 ? wrap : -wrap);
        };
        struct Pend4 { uint2 keys; int q[4], old[4]; };
        // (paired 16-byte key loads, as in the gradient gather, left this pass
        // unchanged: 193 -> 194 us; it is bound by its LDS atomics)
        for_slice<KI_U, 4>(M, wl, c_lo, c_hi, ldkg,
            [&](const auto& r) {
                const float4 gv = g4_of(r, fmt);
                Pend4 p;
                p.keys = r.q;
                issue(r.q.x & 0xFFFFu, gv.x, p.q[0], p.old[0]);
                issue(r.q.x >> 16, gv.y, p.q[1], p.old[1]);
                issue(r.q.y & 0xFFFFu, gv.z, p.q[2], p.old[2]);
                issue(r.q.y >> 16, gv.w, p.q[3], p.old[3]);
                return p;
            },
            [&](uint64_t, const Pend4& p) {
                settle(p.keys.x & 0xFFFFu, p.q[0], p.old[0]);
                settle(p.keys.x >> 16, p.q[1], p.old[1]);
                settle(p.keys.y & 0xFFFFu, p.q[2], p.old[2]);
                settle(p.keys.y >> 16, p.q[3], p.old[3]);
            },
            [&](uint64_t i) {
                int q, old;
                const uint32_t key = keys[i];
                issue(key, g1(i), q, old);
                settle(key, q, old);
            });
        __syncthreads();
        constexpr int RU = 4;   // four LDS reads in flight per thread
        for (int i0 = threadIdx.x; i0 < 2 * w; i0 += RU * NP_THREADS) {
            int a[RU];
#pragma unroll
            for (int q = 0; q < RU; ++q)
                if (i0 + q * NP_THREADS < 2 * w) a[q] = acc32[i0 + q * NP_THREADS];
#pragma unroll
            for (int q = 0; q < RU; ++q)
                if (i0 + q * NP_THREADS < 2 * w)
                    __builtin_nontemporal_store(ldexpf((float)a[q], -S), row + i0 + q * NP_THREADS);
        }
    }
}

// dL/dw_i = g_i H[bits_i] + R[bits_i]; the 8-byte window [lo8, lo8 + w8) of (H, R) sits
// in LDS.  The first workgroup of each matrix also finishes dL/dC^(0); every
// workgroup clears a slice of G for the next backward.
template <bool G16, bool O16>
__global__ void __launch_bounds__(NP_THREADS) k_gather_grad(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float2 hw[2 * W8];
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    const DevState* st = ws.st;
    const int lo = st->lo8, w = st->w8;
    const float2* HR = ws.HR;
    if (wl == 0 && (int)(threadIdx.x >> 6) < M.k) {
        // dL/dC^(0) = (1/tau) sum of the t = 1 partials + the terms that bypass
        // the softmax; wave j takes centroid j (one wave doing all k had held
        // this workgroup back by about 3 us, and with it the whole pass)
        const int T = st->teff, k = M.k, j = threadIdx.x >> 6, lane = threadIdx.x & 63;
        const float* p1 = ws.bpart + (size_t)1 * T_WG * PSTRIDE;
        const float* p0 = ws.bpart;
        const float x = wave_sum(tpart_rows(p1, lane, j));
        const float e = wave_sum(tpart_rows(p0, lane, k + j));
        if (lane == 0) {
            float gc = x * b.inv_tau;
            if (T == 1) gc += e * b.inv_tau;
            if (!(ws.shist[KMAX + j] > 0.f)) gc += ws.ghist[KMAX + j];
            M.gc[j] = gc;
        }
    }
    {
        const uint32_t per = (NKEYS + M.wg_count - 1) / M.wg_count;
        const uint32_t u0 = wl * per, u1 = min((uint32_t)NKEYS, u0 + per);
        for (uint32_t u = u0 + threadIdx.x; u < u1; u += NP_THREADS) ws.G[u] = 0.f;
    }
    fill_lds<2 * W8, NP_THREADS>(hw, HR, 2 * w, [&](int i) {
        const int s = i >= w;
        return (s << 15) | (lo + i - s * w);
    });
    __syncthreads();
    auto look = [&](uint32_t key) -> float2 {   // one flat load per lookup, as in k_gather_wt
        const uint32_t d = (key & 0x7FFFu) - (uint32_t)lo;
        const bool in = d < (uint32_t)w;
        float2 v = hw[(key >> 15) * w + (in ? d : 0u)];
        if (!in) v = HR[key];
        return v;
    };
    auto dw4 = [&](uint32_t k0, uint32_t k1, uint32_t k2, uint32_t k3, float4 gv) {
        const float2 h0 = look(k0), h1 = look(k1), h2 = look(k2), h3 = look(k3);
        return make_float4(fmaf(gv.x, h0.x, h0.y), fmaf(gv.y, h1.x, h1.y),
                           fmaf(gv.z, h2.x, h2.y), fmaf(gv.w, h3.x, h3.y));
    };
    const uint16_t* keys = M.keys;
    const float* g = M.g;
    const uint16_t* gh = reinterpret_cast<const uint16_t*>(M.g);   // G16: 16-bit patterns
    const int fmt = M.fmt;
    auto g1 = [&](uint64_t i) { return G16 ? grad_value(gh[i], fmt) : g[i]; };
    auto dw = [&](uint32_t key, float gv) {
        const float2 h = look(key);
        return fmaf(gv, h.x, h.y);
    };
    float* out = M.gw;
    uint16_t* outh = reinterpret_cast<uint16_t*>(M.gw);           // O16: 16-bit patterns
    auto packed4 = [&](const KeysH4& r) {   // four 16-bit results from four 16-bit gradients
        const float4 o = dw4(r.q.x & 0xFFFFu, r.q.x >> 16, r.q.y & 0xFFFFu, r.q.y >> 16, g4_of(r, fmt));
        return make_uint2(to_half_bits(o.x, fmt) | (to_half_bits(o.y, fmt) << 16),
                          to_half_bits(o.z, fmt) | (to_half_bits(o.w, fmt) << 16));
    };
    if constexpr (G16 && O16) {
        // 16-byte loads and stores, 8 weights per lane and group: with 8-byte
        // ones (4 weights) this pass ran at 4.4 TB/s, with these at 5.4 TB/s
        for_slice<GG16_U, 8, true>(M, wl, 0, 0,
            [&](uint64_t i, auto) { return KeysH8{ld_u4_nt(keys + i), ld_u4_nt(gh + i)}; },
            [&](const KeysH8& r) {
                const uint2 a = packed4(KeysH4{make_uint2(r.q.x, r.q.y), make_uint2(r.g.x, r.g.y)});
                const uint2 c = packed4(KeysH4{make_uint2(r.q.z, r.q.w), make_uint2(r.g.z, r.g.w)});
                return make_uint4(a.x, a.y, c.x, c.y);
            },
            [&](uint64_t i, uint4 o) { st_u4_nt(outh + i, o); },
            [&](uint64_t i) { outh[i] = (uint16_t)to_half_bits(dw(keys[i], g1(i)), fmt); });
        return;
    }
    // A full tile with fp32 dL/dW~: the keys of two groups come in one 16-byte
    // load per lane (lanes 0-31 the first group's 256 keys of this wave, lanes
    // 32-63 the second's) and reach the lanes that use them through
    // ds_bpermute (key_half), so that no lane loads its keys 8 bytes at a
    // time: 340 -> 325 us on the decoder layer (5.95 -> 6.22 TB/s).
    constexpr int GGU = 8;   // groups of 4 weights per lane and tile
    auto full_kp = [&](uint64_t b0, auto) {
        constexpr uint64_t STEP = 4 * NP_THREADS;
        const int lane = threadIdx.x & 63;
        const uint64_t i0 = b0 + 4 * (uint64_t)threadIdx.x;
        const uint64_t seg = b0 + 256 * (uint64_t)(threadIdx.x >> 6) + 8 * (uint64_t)(lane & 31) + (uint64_t)(lane >> 5) * STEP;
        uint4 kq[GGU / 2];
        float4 gv[GGU];
#pragma unroll
        for (int p = 0; p < GGU / 2; ++p) kq[p] = ld_u4_nt(keys + seg + 2 * p * STEP);
#pragma unroll
        for (int u = 0; u < GGU; ++u) gv[u] = ld_f4_nt(g + i0 + u * STEP);
        __builtin_amdgcn_sched_barrier(0);
        const int sa = (lane >> 1) << 2, sb = (32 + (lane >> 1)) << 2;   // source lanes, byte addresses
        const bool odd = lane & 1;
        decltype(dw4(0u, 0u, 0u, 0u, float4{})) o[GGU];
#pragma unroll
        for (int p = 0; p < GGU / 2; ++p) {
            const uint2 ka = key_half(kq[p], sa, odd), kb = key_half(kq[p], sb, odd);
            o[2 * p] = dw4(ka.x & 0xFFFFu, ka.x >> 16, ka.y & 0xFFFFu, ka.y >> 16, gv[2 * p]);
            o[2 * p + 1] = dw4(kb.x & 0xFFFFu, kb.x >> 16, kb.y & 0xFFFFu, kb.y >> 16, gv[2 * p + 1]);
        }
#pragma unroll
        for (int u = 0; u < GGU; ++u) {
            if constexpr (O16)
                st_u2_nt(outh + i0 + u * STEP,
                         make_uint2(to_half_bits(o[u].x, fmt) | (to_half_bits(o[u].y, fmt) << 16),
                                    to_half_bits(o[u].z, fmt) | (to_half_bits(o[u].w, fmt) << 16)));
            else st_f4_nt(out + i0 + u * STEP, o[u]);
        }
    };
    auto full_sel = [&]() {
        if constexpr (!G16) return full_kp;
        else return nullptr;
    };
    for_slice<GGU, 4, true>(M, wl, 0, 0,
        [&](uint64_t i, auto) {
            if constexpr (G16) return KeysH4{ld_u2_nt(keys + i), ld_u2_nt(gh + i)};
            else return KeysG4{ld_u2_nt(keys + i), ld_f4_nt(g + i)};
        },
        [&](const auto& r) {   // the stored form: float4, or (O16) four packed 16-bit values
            const float4 o = dw4(r.q.x & 0xFFFFu, r.q.x >> 16, r.q.y & 0xFFFFu, r.q.y >> 16, g4_of(r, fmt));
            if constexpr (O16)
                return make_uint2(to_half_bits(o.x, fmt) | (to_half_bits(o.y, fmt) << 16),
                                  to_half_bits(o.z, fmt) | (to_half_bits(o.w, fmt) << 16));
            else return o;
        },
        [&](uint64_t i, const auto& o) {
            if constexpr (O16) st_u2_nt(outh + i, o);
            else st_f4_nt(out + i, o);
        },
        [&](uint64_t i) {
            const float v = dw(keys[i], g1(i));
            if constexpr (O16) outh[i] = (uint16_t)to_half_bits(v, fmt);
            else out[i] = v;
        },
        full_sel());
}

// ----------------------------------------------------------------------------
// palettization: the lookup table of k entries and a b-bit index per weight

// Nearest lookup-table entry for every pattern: fp32 distance |v - lut_j|,
// lowest entry on ties; non-finite patterns get 0.  Grid (NKEYS / 256, count).
// The table of the launch's matrix mi: the allocation-free entry point's array
// (single-matrix launches), or the matrix's own workspace region.
__device__ __forceinline__ uint8_t* pal_table(const BatchArgs& b, const MatArgs& M) {
    return b.pal_tab ? b.pal_tab : carve_workspace(M.wsb, M.max_iter).pidx;
}

__global__ void __launch_bounds__(256) k_pal_table(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float lut[KMAX];
    const MatArgs& M = b.m[blockIdx.y];
    uint8_t* const tbl = pal_table(b, M);
    if (threadIdx.x < M.k) lut[threadIdx.x] = M.c_in[threadIdx.x];
    __syncthreads();
    const uint32_t u = blockIdx.x * 256 + threadIdx.x;
    uint32_t best = 0;
    if (key_finite(u, M.fmt)) {
        const float v = key_value(u, M.fmt);
        float bd = fabsf(v - lut[0]);
        for (int j = 1; j < M.k; ++j) {
            const float d = fabsf(v - lut[j]);
            if (d < bd) { bd = d; best = (uint32_t)j; }
        }
    }
    tbl[u] = (uint8_t)best;
}

// Packed indices: index i occupies bits [B i, B i + B) of a little-endian bit
// stream.  A thread packs a group of 32 weights into B 32-bit words (4 B bytes
// at byte 4 B g for group g); the per-pattern index table (64 KiB) sits in LDS.
// The matrix's last, partial group and unaligned buffers are written byte by
// byte, never past the ceil(n B / 8) output bytes.  A matrix's workgroups
// [b.wg_begin[mi], b.wg_begin[mi] + wg_count) take its groups round-robin, 1024 at a time.
template <int B>
__global__ void __launch_bounds__(1024) k_palettize(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ uint4 tbl4[NKEYS / 16];
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    const uint4* src = reinterpret_cast<const uint4*>(pal_table(b, M));
    fill_lds<NKEYS / 16, 1024>(tbl4, src, NKEYS / 16, [](int i) { return i; });   // blockDim.x = 1024
    __syncthreads();
    const uint8_t* tbl = reinterpret_cast<const uint8_t*>(tbl4);
    const uint16_t* keys = M.keys;
    uint32_t* out32 = reinterpret_cast<uint32_t*>(M.wt);
    uint8_t* out8 = reinterpret_cast<uint8_t*>(M.wt);
    const uint64_t n = M.n;
    const uint64_t groups = (n + 31) / 32;
    const uint64_t nbytes = (n * B + 7) / 8;
    for (uint64_t gi = (uint64_t)wl * blockDim.x + threadIdx.x; gi < groups;
         gi += (uint64_t)M.wg_count * blockDim.x) {
        const uint64_t base = gi * 32;
        uint32_t w[B];
#pragma unroll
        for (int q = 0; q < B; ++q) w[q] = 0u;
        auto put = [&](int t, uint32_t idx) {   // t is a compile-time constant after unrolling
            const int pos = t * B;
            w[pos >> 5] |= idx << (pos & 31);
            if ((pos & 31) + B > 32) w[(pos >> 5) + 1] |= idx >> (32 - (pos & 31));
        };
        if (base + 32 <= n && M.vec) {
            uint4 q[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) q[r] = ld_u4(keys + base + 8 * r);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const uint32_t x[4] = {q[r].x, q[r].y, q[r].z, q[r].w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    put(8 * r + 2 * h, tbl[x[h] & 0xFFFFu]);
                    put(8 * r + 2 * h + 1, tbl[x[h] >> 16]);
                }
            }
#pragma unroll
            for (int q2 = 0; q2 < B; ++q2) __builtin_nontemporal_store(w[q2], out32 + gi * B + q2);
        } else {
#pragma unroll
            for (int t = 0; t < 32; ++t)
                if (base + t < n) put(t, tbl[keys[base + t]]);
            const uint64_t b0 = gi * 4 * B;
#pragma unroll
            for (int q2 = 0; q2 < 4 * B; ++q2)
                if (b0 + q2 < nbytes) out8[b0 + q2] = (uint8_t)(w[q2 >> 2] >> (8 * (q2 & 3)));
        }
    }
}

// ----------------------------------------------------------------------------
// Distinct patterns and the inverse index: the unique-value list and the
// per-weight index list of the uniquification (Sec. 2.2), in ascending order
// of the 16-bit key (the order np.unique gives)

// rank[u] = number of occupied patterns (count > 0) below u, for every u.  For
// an occupied u that is its position in the sorted list of distinct patterns,
// written to M.uniq when given.  One 1024-thread block per matrix, grid
// (1, count); thread t ranks the patterns [64 t, 64 t + 64).
__global__ void __launch_bounds__(1024) k_rank(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ unsigned long long occ[NKEYS / 64];   // bit e of word t: pattern 64 t + e occupied
    __shared__ uint32_t wtot[1024 / 64];
    const MatArgs& M = b.m[blockIdx.y];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    // byte m of the bitmap (patterns 8 m .. 8 m + 7) from two 16-byte loads of
    // counts; m = 1024 i + t keeps every load contiguous across the wave
    const uint4* c4 = reinterpret_cast<const uint4*>(ws.counts);
    uint4 q[16];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        q[2 * i] = c4[2 * (1024 * i + t)];
        q[2 * i + 1] = c4[2 * (1024 * i + t) + 1];
    }
    uint8_t* occ8 = reinterpret_cast<uint8_t*>(occ);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint4 a = q[2 * i], c = q[2 * i + 1];
        occ8[1024 * i + t] =
            (uint8_t)((uint32_t)(a.x != 0u) | (uint32_t)(a.y != 0u) << 1 | (uint32_t)(a.z != 0u) << 2 |
                      (uint32_t)(a.w != 0u) << 3 | (uint32_t)(c.x != 0u) << 4 | (uint32_t)(c.y != 0u) << 5 |
                      (uint32_t)(c.z != 0u) << 6 | (uint32_t)(c.w != 0u) << 7);
    }
    __syncthreads();
    const unsigned long long bits = occ[t];
    const uint32_t pc = (uint32_t)__popcll(bits);
    const uint32_t incl = wave_incl_scan(pc);
    if (lane == 63) wtot[wave] = incl;
    __syncthreads();
    uint32_t base = incl - pc;   // occupied patterns below 64 t
    for (int w = 0; w < wave; ++w) base += wtot[w];
    // the thread's 64 ranks, 8 per 16-byte store (pattern 2 j in the low half
    // of word j); a rank never exceeds 65,535
    uint4* rk = reinterpret_cast<uint4*>(ws.rank + 64 * t);
    uint32_t r = base;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
        uint32_t h[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = 8 * g + 2 * j;
            const uint32_t r0 = r;
            r += (uint32_t)(bits >> e) & 1u;
            h[j] = r0 | (r << 16);
            r += (uint32_t)(bits >> (e + 1)) & 1u;
        }
        rk[g] = make_uint4(h[0], h[1], h[2], h[3]);
    }
    if (M.uniq) {
        unsigned long long x = bits;
        uint32_t ru = base;
        while (x) {
            M.uniq[ru++] = (uint16_t)(64 * t + __builtin_ctzll(x));
            x &= x - 1;
        }
    }
}

// inverse[i] = rank[bits_i]: the position of w_i's pattern among the distinct
// patterns.  The whole rank table (128 KiB) is loaded into LDS; no window.
// Matrices of the launch without an inverse output (M.wt null) skip the pass.
__global__ void __launch_bounds__(NP_THREADS) k_inverse(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ uint4 rk4[NKEYS * sizeof(uint16_t) / sizeof(uint4)];
    const int mi = np_matrix(b);
    const MatArgs M = np_args(b, mi);
    if (!M.wt) return;   // the same for the whole workgroup
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const uint32_t wl = blockIdx.x - b.wg_begin[mi];
    const uint4* src = reinterpret_cast<const uint4*>(ws.rank);
    constexpr int NV = NKEYS * sizeof(uint16_t) / sizeof(uint4);
    fill_lds<NV, NP_THREADS>(rk4, src, NV, [](int i) { return i; });
    __syncthreads();
    const uint16_t* rk = reinterpret_cast<const uint16_t*>(rk4);
    const uint16_t* keys = M.keys;
    uint16_t* out = reinterpret_cast<uint16_t*>(M.wt);
    auto pair = [&](uint32_t x) { return (uint32_t)rk[x & 0xFFFFu] | ((uint32_t)rk[x >> 16] << 16); };
    for_slice<8, 8>(M, wl, 0, 0,
        [&](uint64_t i, auto) { return Keys8{ld_u4_nt(keys + i)}; },
        [&](const Keys8& r) { return make_uint4(pair(r.q.x), pair(r.q.y), pair(r.q.z), pair(r.q.w)); },
        [&](uint64_t i, uint4 o) { st_u4_nt(out + i, o); },
        [&](uint64_t i) { out[i] = rk[keys[i]]; });
}

// ----------------------------------------------------------------------------
// backward table phase

// The backward's first table quantities, from the keyed-sum partial rows:
//   gamma_j = sum_u G_u a^(T)_uj                                   (= dL/dC^(T)_j)
//   E_j     = sum_u G_u a^(T)_uj (C^(T)_j - Tab_u) sgn(v_u - C^(T-1)_j)
// (a^(T) built from C^(T-1); E without the 1/tau).  Both are linear in the
// keyed sums G_u, so G_u is never assembled: a thread sums one window
// pattern's entries over a chunk of GT_ROWS partial rows (blockIdx.y) and
// adds that partial sum times the pattern's terms.  The last blockIdx.y takes
// what the keyed-sum pass added to the global G instead (patterns outside the
// window, values above its fixed-point limit, wrap corrections), over all
// 65,536 patterns.  Block totals are added with float atomics into the 64 rows
// of the backward's first partial block, which k_keyed_grad clears.
// (Summing the rows into G first, then
// a table kernel over G, took one launch more.)  Grid (MERGE_X, row chunks +
// 1, count).
constexpr int MERGE_X = 2 * W4 / MERGE_THREADS;
// Rows per chunk here: a pattern's terms are evaluated once per chunk, so
// larger chunks than the histogram merge's (one for a decoder layer's
// matrices, of at most 57 rows each).
constexpr int GT_ROWS = 64;
template <int K>
__global__ void __launch_bounds__(MERGE_THREADS) k_grad_top(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    static_assert(MERGE_THREADS == T_THREADS, "block_total sums over T_THREADS");
    __shared__ float red[BLOCK_TOTAL_LDS(2 * K)];
    constexpr int GPER = (NKEYS + MERGE_X * MERGE_THREADS - 1) / (MERGE_X * MERGE_THREADS);
    const MatArgs& M = b.m[blockIdx.z];
    // the arguments in one wait, then the window and C^(T-1), C^(T) in one
    // more (read where they are used, they had cost five round trips before
    // the first row load)
    const int fmt = M.fmt, wg_count = (int)M.wg_count;
    const float s2 = b.s2;
    const uint32_t gy = gridDim.y;
    asm volatile("" ::"s"(fmt), "s"(wg_count), "s"(s2), "s"(gy), "s"(M.wsb), "s"(M.max_iter));
    const bool gblock = blockIdx.y == gy - 1;
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const DevState* st = ws.st;
    const int kmode = st->kmode, w4 = st->w4, lo4 = st->lo4, w8 = st->w8, lo8 = st->lo8;
    float c0[K], c1[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c0[j] = ws.cfin[j]; c1[j] = ws.cfin[KMAX + j]; }
    float gv[GPER];
    uint32_t key[GPER];
#pragma unroll
    for (int q = 0; q < GPER; ++q) { gv[q] = 0.f; key[q] = 0u; }
    if (gblock) {
        // the global G: GPER patterns per thread
#pragma unroll
        for (int q = 0; q < GPER; ++q) {
            const uint32_t u = (q * MERGE_X + blockIdx.x) * MERGE_THREADS + threadIdx.x;
            key[q] = u;
            if (u < (uint32_t)NKEYS) gv[q] = ws.G[u];
        }
    } else {
        const bool wide = kmode == KEYED_U64;
        const int w = wide ? w8 : w4, lo = wide ? lo8 : lo4;
        const int r0 = blockIdx.y * GT_ROWS;
        const int r1 = min(wg_count, r0 + GT_ROWS);
        if (r0 >= r1 || (int)(blockIdx.x * MERGE_THREADS) >= 2 * w) return;   // the same for the block
        const int i = blockIdx.x * MERGE_THREADS + threadIdx.x;
        if (i < 2 * w) {
            const float* part = reinterpret_cast<const float*>(ws.part) + i;
            float x[GT_ROWS];                      // every row's value in flight at once
#pragma unroll
            for (int q = 0; q < GT_ROWS; ++q) x[q] = r0 + q < r1 ? part[(size_t)(r0 + q) * ROW4] : 0.f;
#pragma unroll
            for (int h = GT_ROWS / 2; h > 0; h /= 2)   // pairwise sum
#pragma unroll
                for (int q = 0; q < h; ++q) x[q] += x[q + h];
            const int sg = i >= w;
            gv[0] = x[0];
            key[0] = (uint32_t)((sg << 15) | (lo + i - sg * w));
        }
    }
    EDKM_STAMP_MARK(b, 2);   // rows summed (G loaded)
    int nz = 0;
#pragma unroll
    for (int q = 0; q < GPER; ++q) nz |= gv[q] != 0.f;
    if (!__syncthreads_or(nz)) return;   // nothing to add in this block
    float acc[2 * K];
#pragma unroll
    for (int j = 0; j < 2 * K; ++j) acc[j] = 0.f;
#pragma unroll
    for (int q = 0; q < GPER; ++q) {
        if (gv[q] == 0.f || !key_finite(key[q], fmt)) continue;
        const float v = key_value(key[q], fmt);
        float a[K], d[K], c1m;
        attn_row_sel<K>(v, c0, s2, a, c1, c1m);
        centroid_dev<K>(a, c1, c1m, d);
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const float ga = gv[q] * a[j];
            acc[j] += ga;
            acc[K + j] = fmaf(ga * d[j], sgnf(v - c0[j]), acc[K + j]);
        }
    }
    EDKM_STAMP_MARK(b, 3);   // patterns done
    const float tot = block_total<2 * K>(acc, red);
    EDKM_STAMP_MARK(b, 4);   // block summed
    if (threadIdx.x < 2 * K && tot != 0.f) {
        const int row = (blockIdx.x + 7 * blockIdx.y) % T_WG;   // spread over the rows
        atomicAdd(&ws.bpart[(size_t)row * PSTRIDE + threadIdx.x], tot);
    }
}

// Iteration t = T..1 of the backward: gamma = dL/dC^(t), then per occupied
// pattern
//   alpha_j = gamma_j (v_u - C^(t)_j) / S^(t)_j,  abar = sum_j a_uj alpha_j,
//   delta_j = a_uj (alpha_j - abar),
//   R_u    += sum_j a_uj gamma_j / S^(t)_j - (1/tau) sum_j delta_j sgn(v_u - C^(t-1)_j),
// and partials of sum_u n_u delta_j sgn(v_u - C^(t-1)_j), which (times 1/tau)
// make dL/dC^(t-1).  Grid (T_WG, count).
template <int K>
__global__ void __launch_bounds__(T_THREADS) k_bwd_iter(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float red[BLOCK_TOTAL_LDS(K)];
    __shared__ float gSsh[K], c1sh[K], c0sh[K];
    const MatArgs& M = b.m[blockIdx.y];
    const int t = b.t;
    // the arguments, in one wait (read where they are used, each had cost a
    // round trip of its own), then the executed iteration count with the loads
    const int max_iter = M.max_iter, fmt = M.fmt;
    const float s2 = b.s2, inv_tau = b.inv_tau;
    asm volatile("" ::"s"(max_iter), "s"(fmt), "s"(t), "s"(s2), "s"(inv_tau), "s"(M.wsb));
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const DevState* st = ws.st;
    const int T = st->teff;
    // Every load first, none waiting for T: the per-pattern inputs, the
    // partial blocks (columns [0, 2K) of block 0 -- k_grad_top's, used at
    // t = T and t = T - 1 -- and [0, K) of block t + 1), and the k-vectors of
    // iterations t - 1, t, t + 1.
    uint32_t n4[T_KPT];
    float R4[T_KPT], H4[T_KPT];
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) {
        const int u = table_key(r);
        n4[r] = ws.counts[u];
        R4[r] = t < max_iter ? ws.R[u] : 0.f;
        H4[r] = t == 1 ? ws.H[u] : 0.f;
    }
    PartCols<4 * K> pc;
    const float* b0 = ws.bpart;
    const float* bn = t < max_iter ? ws.bpart + (size_t)(t + 1) * T_WG * PSTRIDE : nullptr;
    pc.load([&](int c) -> const float* {
        return c < 2 * K ? b0 + c : (c < 3 * K && bn ? bn + (c - 2 * K) : nullptr);
    });
    float hc1 = 0.f, hc0 = 0.f, hS = 0.f, hS1 = 0.f, hg1 = 0.f;
    if (threadIdx.x < K) {
        const int j = threadIdx.x;
        hc1 = ws.chist[t * KMAX + j];
        hc0 = ws.chist[(t - 1) * KMAX + j];
        hS = ws.shist[t * KMAX + j];
        if (t < max_iter) { hS1 = ws.shist[(t + 1) * KMAX + j]; hg1 = ws.ghist[(t + 1) * KMAX + j]; }
    }
    EDKM_STAMP_MARK(b, 2);   // loads issued
    pc.stage(red);
    if (t > T) return;
    const bool lead = blockIdx.x == 0;
    if (threadIdx.x < K) {
        const int j = threadIdx.x;
        float gm;
        if (t == T) {
            gm = PartCols<4 * K>::total(red, j);
        } else {
            gm = PartCols<4 * K>::total(red, 2 * K + j) * inv_tau;
            if (t + 1 == T) gm += PartCols<4 * K>::total(red, K + j) * inv_tau;
            if (!(hS1 > 0.f)) gm += hg1;
        }
        c1sh[j] = hc1;
        c0sh[j] = hc0;
        gSsh[j] = hS > 0.f ? gm / hS : 0.f;
        if (lead) ws.ghist[t * KMAX + j] = gm;
    }
    __syncthreads();
    EDKM_STAMP_MARK(b, 3);   // partial blocks summed, gamma formed
    float c1[K], c0[K], gS[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c1[j] = c1sh[j]; c0[j] = c0sh[j]; gS[j] = gSsh[j]; }
    float acc[K];
#pragma unroll
    for (int j = 0; j < K; ++j) acc[j] = 0.f;
#pragma unroll
    for (int r = 0; r < T_KPT; ++r) {
        const int u = table_key(r);
        const uint32_t n = n4[r];
        if (n == 0u) continue;
        if (!key_finite(u, fmt)) {
            if (t == 1) ws.HR[u] = make_float2(__builtin_nanf(""), __builtin_nanf(""));
            continue;
        }
        const float v = key_value(u, fmt);
        float a[K], dev[K], cm;
        attn_row_sel<K>(v, c0, s2, a, c1, cm);
        const float direct = softmax_dev<K>(v, a, gS, c1, cm, dev);
        const float nf = (float)n;
        float r_ = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const float dl = a[j] * dev[j] * sgnf(v - c0[j]);
            r_ += dl;
            acc[j] = fmaf(nf, dl, acc[j]);
        }
        const float Ru = fmaf(-r_, inv_tau, direct) + (t != T ? R4[r] : 0.f);
        if (t == 1) ws.HR[u] = make_float2(H4[r], Ru);
        else ws.R[u] = Ru;
    }
    EDKM_STAMP_MARK(b, 4);   // patterns done
    const float tot = block_total<K>(acc, red);
    EDKM_STAMP_MARK(b, 5);   // block summed
    if (threadIdx.x < K) ws.bpart[((size_t)t * T_WG + blockIdx.x) * PSTRIDE + threadIdx.x] = tot;
}

// ----------------------------------------------------------------------------
// dense (non-uniquified) comparison path: one attention row per weight

__device__ __forceinline__ bool dense_range(const MatArgs& M, uint64_t& beg, uint64_t& end) {
    beg = (uint64_t)blockIdx.x * M.chunk;
    end = min(M.n, beg + M.chunk);
    return beg < end;
}

// Fixed-order sum of the first nrow dense partial rows, columns [c0, c0+ncol),
// by one block of 1024 threads; result in out[0..ncol) (LDS).
__device__ __forceinline__ void reduce_dparts(const float* part, int nrow, int c0, int ncol,
                                              float* scratch /*16*32*/, float* out) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int j = 0; j < ncol; ++j) {
        float x = threadIdx.x < nrow ? part[threadIdx.x * PSTRIDE + c0 + j] : 0.f;
        x = wave_sum(x);
        if (lane == 0) scratch[wave * PSTRIDE + j] = x;
    }
    __syncthreads();
    if (threadIdx.x < ncol) {
        float s = 0.f;
        for (int w = 0; w < 16; ++w) s += scratch[w * PSTRIDE + threadIdx.x];
        out[threadIdx.x] = s;
    }
    __syncthreads();
}

template <int K>
__global__ void __launch_bounds__(D_THREADS) k_dense_iter(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float tot[2 * K];
    __shared__ float scratch[D_THREADS / 64 * 2 * K];
    __shared__ float csh[K];
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int t = b.t;
    if (t > 1 && ws.st->conv) return;
    if (threadIdx.x < K) csh[threadIdx.x] = t == 1 ? M.c_in[threadIdx.x] : ws.chist[(t - 1) * KMAX + threadIdx.x];
    __syncthreads();
    float c[K];
#pragma unroll
    for (int j = 0; j < K; ++j) c[j] = csh[j];
    float acc[2 * K];
#pragma unroll
    for (int j = 0; j < 2 * K; ++j) acc[j] = 0.f;
    uint64_t beg, end;
    dense_range(M, beg, end);
    for (uint64_t i = beg + threadIdx.x; i < end; i += D_THREADS) {
        const uint32_t key = M.keys[i];
        if (!key_finite(key, M.fmt)) continue;
        const float v = key_value(key, M.fmt);
        float a[K];
        float unused;
        const float r = attn_row_dense_un<K>(v, c, b.s2, a, c, unused);   // normalised below
        const float rv = r * v;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            acc[j] = fmaf(a[j], r, acc[j]);
            acc[K + j] = fmaf(a[j], rv, acc[K + j]);
        }
    }
    block_sum<2 * K, D_THREADS>(acc, scratch, tot);
    if (threadIdx.x < 2 * K) ws.dpart[(size_t)blockIdx.x * PSTRIDE + threadIdx.x] = tot[threadIdx.x];
}

// One block: C^(t) from the dense partials, history, early stop.
template <int K>
__global__ void __launch_bounds__(1024) k_dense_fin(BatchArgs b, int nrow) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float scratch[16 * PSTRIDE];
    __shared__ float tot[2 * K];
    __shared__ int stop;
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    DevState* st = ws.st;
    const int t = b.t;
    if (t > 1 && st->conv) return;
    reduce_dparts(ws.dpart, nrow, 0, 2 * K, scratch, tot);
    if (threadIdx.x == 0) stop = 0;
    __syncthreads();
    if (threadIdx.x < K) {
        const int j = threadIdx.x;
        const float cprev = t == 1 ? M.c_in[j] : ws.chist[(t - 1) * KMAX + j];
        if (t == 1) { ws.chist[j] = cprev; ws.shist[j] = 0.f; }
        const float S = tot[j], P = tot[K + j];
        const float cn = S > 0.f ? P / S : cprev;
        ws.chist[t * KMAX + j] = cn;
        ws.shist[t * KMAX + j] = S;
        if (!(fabsf(cn - cprev) <= b.eps)) atomicOr(&stop, 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        if (b.eps > 0.f && stop == 0) { st->conv = 1; st->teff = t; }
        else { st->conv = 0; st->teff = t; }
    }
}

template <int K>
__global__ void __launch_bounds__(D_THREADS) k_dense_out(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int T = ws.st->teff;
    __shared__ float c1sh[K], c0sh[K];
    if (threadIdx.x < K) {
        c1sh[threadIdx.x] = ws.chist[T * KMAX + threadIdx.x];
        c0sh[threadIdx.x] = ws.chist[(T - 1) * KMAX + threadIdx.x];
    }
    __syncthreads();
    float c1[K], c0[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c1[j] = c1sh[j]; c0[j] = c0sh[j]; }
    if (blockIdx.x == 0) {
        if (threadIdx.x < K) M.c_out[threadIdx.x] = ws.chist[T * KMAX + threadIdx.x];
        if (threadIdx.x == 0 && M.iters_out) *M.iters_out = T;
    }
    uint64_t beg, end;
    dense_range(M, beg, end);
    for (uint64_t i = beg + threadIdx.x; i < end; i += D_THREADS) {
        const uint32_t key = M.keys[i];
        float wv;
        float a[K];
        if (key_finite(key, M.fmt)) {
            const float v = key_value(key, M.fmt);
            float unused;
            attn_row_dense<K>(v, c0, b.s2, a, c0, unused);
            wv = 0.f;
#pragma unroll
            for (int j = 0; j < K; ++j) wv = fmaf(a[j], c1[j], wv);
        } else {
            wv = __builtin_nanf("");
#pragma unroll
            for (int j = 0; j < K; ++j) a[j] = __builtin_nanf("");
        }
        if (b.out_half) reinterpret_cast<uint16_t*>(M.wt)[i] = (uint16_t)to_half_bits(wv, M.fmt);
        else reinterpret_cast<float*>(M.wt)[i] = wv;
        if (M.attn) {
#pragma unroll
            for (int j = 0; j < K; ++j) M.attn[i * K + j] = a[j];
        }
    }
}

// Dense backward, direct use of A^(T): dL/dw_i = g_i H_i, and partials of gamma and E.
template <int K>
__global__ void __launch_bounds__(D_THREADS) k_dense_btop(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float tot[2 * K];
    __shared__ float scratch[D_THREADS / 64 * 2 * K];
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int T = ws.st->teff;
    __shared__ float c1sh[K], c0sh[K];
    if (threadIdx.x < K) {
        c1sh[threadIdx.x] = ws.chist[T * KMAX + threadIdx.x];
        c0sh[threadIdx.x] = ws.chist[(T - 1) * KMAX + threadIdx.x];
    }
    __syncthreads();
    float c1[K], c0[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c1[j] = c1sh[j]; c0[j] = c0sh[j]; }
    float acc[2 * K];
#pragma unroll
    for (int j = 0; j < 2 * K; ++j) acc[j] = 0.f;
    uint64_t beg, end;
    dense_range(M, beg, end);
    for (uint64_t i = beg + threadIdx.x; i < end; i += D_THREADS) {
        const uint32_t key = M.keys[i];
        if (!key_finite(key, M.fmt)) { M.gw[i] = __builtin_nanf(""); continue; }
        const float v = key_value(key, M.fmt);
        const float g = M.g[i];
        float a[K], d[K], c1m;
        attn_row_dense<K>(v, c0, b.s2, a, c1, c1m);
        centroid_dev<K>(a, c1, c1m, d);
        float h = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const float q = a[j] * d[j] * sgnf(v - c0[j]);
            h += q;
            acc[j] = fmaf(g, a[j], acc[j]);
            acc[K + j] = fmaf(g, q, acc[K + j]);
        }
        M.gw[i] = -g * h * b.inv_tau;
    }
    block_sum<2 * K, D_THREADS>(acc, scratch, tot);
    if (threadIdx.x < 2 * K) ws.dpart[(size_t)blockIdx.x * PSTRIDE + threadIdx.x] = tot[threadIdx.x];
}

// Dense backward iteration t (reads gamma^(t) from ghist).
template <int K>
__global__ void __launch_bounds__(D_THREADS) k_dense_biter(BatchArgs b) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float tot[K];
    __shared__ float scratch[D_THREADS / 64 * K];
    __shared__ float c1sh[K], c0sh[K], gSsh[K];
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int T = ws.st->teff;
    const int t = b.t;
    if (t > T) return;
    if (threadIdx.x < K) {
        const int j = threadIdx.x;
        c1sh[j] = ws.chist[t * KMAX + j];
        c0sh[j] = ws.chist[(t - 1) * KMAX + j];
        const float S = ws.shist[t * KMAX + j];
        gSsh[j] = S > 0.f ? ws.ghist[t * KMAX + j] / S : 0.f;
    }
    __syncthreads();
    float c1[K], c0[K], gS[K];
#pragma unroll
    for (int j = 0; j < K; ++j) { c1[j] = c1sh[j]; c0[j] = c0sh[j]; gS[j] = gSsh[j]; }
    float acc[K];
#pragma unroll
    for (int j = 0; j < K; ++j) acc[j] = 0.f;
    uint64_t beg, end;
    dense_range(M, beg, end);
    for (uint64_t i = beg + threadIdx.x; i < end; i += D_THREADS) {
        const uint32_t key = M.keys[i];
        if (!key_finite(key, M.fmt)) continue;
        const float v = key_value(key, M.fmt);
        float a[K], dev[K], cm;
        attn_row_dense<K>(v, c0, b.s2, a, c1, cm);
        const float direct = softmax_dev<K>(v, a, gS, c1, cm, dev);
        float r = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) {
            const float dl = a[j] * dev[j] * sgnf(v - c0[j]);
            r += dl;
            acc[j] += dl;
        }
        M.gw[i] += fmaf(-r, b.inv_tau, direct);
    }
    block_sum<K, D_THREADS>(acc, scratch, tot);
    if (threadIdx.x < K) ws.dpart[(size_t)blockIdx.x * PSTRIDE + threadIdx.x] = tot[threadIdx.x];
}

// One block.  b.t = 0 (after btop): gamma^(T) = dL/dC^(T) and E.  b.t = t in
// T..1 (after biter t): gamma^(t-1) = dL/dC^(t-1); at t = 1 also dL/dC^(0).
template <int K>
__global__ void __launch_bounds__(1024) k_dense_bfin(BatchArgs b, int nrow) {
    EDKM_STAMP_ENTRY(b);
    __shared__ float scratch[16 * PSTRIDE];
    __shared__ float tot[2 * K];
    const MatArgs& M = b.m[0];
    const Ws ws = carve_workspace(M.wsb, M.max_iter);
    const int T = ws.st->teff;
    const int t = b.t;
    if (t == 0) {
        reduce_dparts(ws.dpart, nrow, 0, 2 * K, scratch, tot);
        if (threadIdx.x < K) {
            ws.ghist[T * KMAX + threadIdx.x] = tot[threadIdx.x];
            ws.ehist[threadIdx.x] = tot[K + threadIdx.x] * b.inv_tau;
        }
        return;
    }
    if (t > T) return;
    reduce_dparts(ws.dpart, nrow, 0, K, scratch, tot);
    if (threadIdx.x < K) {
        const int j = threadIdx.x;
        float gm = tot[j] * b.inv_tau;
        if (t == T) gm += ws.ehist[j];
        if (!(ws.shist[t * KMAX + j] > 0.f)) gm += ws.ghist[t * KMAX + j];
        ws.ghist[(t - 1) * KMAX + j] = gm;
        if (t == 1) M.gc[j] = gm;
    }
}

// ----------------------------------------------------------------------------
// Library-owned scratch of the allocation-free palettization: the index table
// of one matrix, one copy per GPU (held until the process ends).  Host code
// never passes the array's name to a kernel (on the host it only names the
// symbol); it uses the device address that hipGetSymbolAddress returns, looked
// up once per device with that device current.

static __device__ __align__(256) uint8_t scratch[NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(uint8_t** out) {
    static std::atomic<uint8_t*> addr[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    uint8_t* p = addr[dev].load(std::memory_order_acquire);
    if (!p) {
        void* q = nullptr;
        e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!q) return hipErrorInvalidSymbol;
        p = static_cast<uint8_t*>(q);
        addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return hipSuccess;
}

// ----------------------------------------------------------------------------
// launch sequences

// Each launch is followed by a check; the name of a failing launch goes to *where.
// An N-sized pass, with the caller's timing events recorded around it if set.
#define EDKM_NPASS(pass, name, kern, grid, block, ...)                                   \
    do {                                                                                 \
        if (ev && ev->start[pass]) { hipError_t e0_ = hipEventRecord(ev->start[pass], s); \
            if (e0_ != hipSuccess) { *where = "hipEventRecord"; return e0_; } }            \
        EDKM_LAUNCH(name, kern, grid, block, __VA_ARGS__);                               \
        if (ev && ev->stop[pass]) { hipError_t e1_ = hipEventRecord(ev->stop[pass], s);   \
            if (e1_ != hipSuccess) { *where = "hipEventRecord"; return e1_; } }            \
    } while (0)

#define EDKM_LAUNCH(name, kern, grid, block, ...)                       \
    do {                                                                  \
        EDKM_STAMP_SLOT(b, name);                                         \
        hipLaunchKernelGGL(kern, grid, block, 0, s, __VA_ARGS__);         \
        hipError_t e_ = hipGetLastError();                                \
        if (e_ != hipSuccess) { *where = name; return e_; }              \
    } while (0)

// Row chunks of `per` rows for a partial-row merge: enough for the matrix of
// the launch with the most N-pass workgroups (one partial row each).
static uint32_t merge_chunks(const BatchArgs& b, int per = MERGE_ROWS) {
    uint32_t rows = 1;
    for (int i = 0; i < b.count; ++i) rows = b.m[i].wg_count > rows ? b.m[i].wg_count : rows;
    return (rows + per - 1) / per;
}

template <int K>
static hipError_t forward_k(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                            const PassEvents* ev) {
    const dim3 tg(T_WG, b.count);
    for (int t = 1; t <= max_t; ++t) {
        b.t = t;
        EDKM_LAUNCH("k_fwd_iter", k_fwd_iter<K>, tg, dim3(T_THREADS), b);
    }
    EDKM_LAUNCH("k_fwd_out", k_fwd_out<K>, tg, dim3(T_THREADS), b);
    EDKM_NPASS(PASS_GATHER_WT, "k_gather_wt", k_gather_wt, dim3(grid_np), dim3(NP_THREADS), b);
    return hipSuccess;
}

template <int K>
static hipError_t backward_k(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                             const PassEvents* ev) {
    const dim3 tg(T_WG, b.count);
    if (b.g_half) EDKM_NPASS(PASS_KEYED_GRAD, "k_keyed_grad", k_keyed_grad<true>, dim3(grid_np), dim3(NP_THREADS), b);
    else EDKM_NPASS(PASS_KEYED_GRAD, "k_keyed_grad", k_keyed_grad<false>, dim3(grid_np), dim3(NP_THREADS), b);
    EDKM_LAUNCH("k_grad_top", k_grad_top<K>, dim3(MERGE_X, merge_chunks(b, GT_ROWS) + 1, b.count),
                dim3(MERGE_THREADS), b);
    for (int t = max_t; t >= 1; --t) {
        b.t = t;
        EDKM_LAUNCH("k_bwd_iter", k_bwd_iter<K>, tg, dim3(T_THREADS), b);
    }
    const dim3 gg(grid_np), gb(NP_THREADS);
    if (b.g_half && b.gw_half) EDKM_NPASS(PASS_GATHER_GRAD, "k_gather_grad", (k_gather_grad<true, true>), gg, gb, b);
    else if (b.g_half) EDKM_NPASS(PASS_GATHER_GRAD, "k_gather_grad", (k_gather_grad<true, false>), gg, gb, b);
    else if (b.gw_half) EDKM_NPASS(PASS_GATHER_GRAD, "k_gather_grad", (k_gather_grad<false, true>), gg, gb, b);
    else EDKM_NPASS(PASS_GATHER_GRAD, "k_gather_grad", (k_gather_grad<false, false>), gg, gb, b);
    return hipSuccess;
}

template <int K>
static hipError_t forward_dense_k(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                  const PassEvents* ev) {
    const int max_t = b.m[0].max_iter;
    for (int t = 1; t <= max_t; ++t) {
        b.t = t;
        EDKM_NPASS(PASS_DENSE_ITER, "k_dense_iter", k_dense_iter<K>, dim3(nwg), dim3(D_THREADS), b);
        EDKM_LAUNCH("k_dense_fin", k_dense_fin<K>, dim3(1), dim3(1024), b, (int)nwg);
    }
    EDKM_LAUNCH("k_dense_out", k_dense_out<K>, dim3(nwg), dim3(D_THREADS), b);
    return hipSuccess;
}

template <int K>
static hipError_t backward_dense_k(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                   const PassEvents* ev) {
    const int max_t = b.m[0].max_iter;
    EDKM_LAUNCH("k_dense_btop", k_dense_btop<K>, dim3(nwg), dim3(D_THREADS), b);
    b.t = 0;
    EDKM_LAUNCH("k_dense_bfin", k_dense_bfin<K>, dim3(1), dim3(1024), b, (int)nwg);
    for (int t = max_t; t >= 1; --t) {
        b.t = t;
        EDKM_NPASS(PASS_DENSE_BITER, "k_dense_biter", k_dense_biter<K>, dim3(nwg), dim3(D_THREADS), b);
        EDKM_LAUNCH("k_dense_bfin", k_dense_bfin<K>, dim3(1), dim3(1024), b, (int)nwg);
    }
    return hipSuccess;
}

// Cached loads for the last IC_KEEP_KEYS keys of a pass's sweeps (spread over
// the launch's matrices in proportion), non-temporal loads before: only the
// end of a sweep, as many keys as fill the 256 MB Infinity Cache, can still be
// there when the next pass starts, and non-temporal loads stream faster
// (histogram of the decoder layer's 202M keys: 74 us all non-temporal, 78 us
// all cached).
constexpr double IC_KEEP_KEYS = 134217728.0;   // 256 MB of 16-bit keys
static void set_keep_frac(BatchArgs& b) {
    double n = 0.0;
    for (int i = 0; i < b.count; ++i) n += (double)b.m[i].n;
    b.keep_frac = n <= IC_KEEP_KEYS ? 1.0f : (float)(IC_KEEP_KEYS / n);
}

#define EDKM_DISPATCH_K(k, fn, ...)            \
    switch (k) {                               \
    case 2: return fn<2>(__VA_ARGS__);         \
    case 4: return fn<4>(__VA_ARGS__);         \
    case 8: return fn<8>(__VA_ARGS__);         \
    case 16: return fn<16>(__VA_ARGS__);       \
    default: return hipErrorInvalidValue;      \
    }

hipError_t launch_init_unique(BatchArgs& b, uint32_t grid_np, hipStream_t s, const char** where,
                              const PassEvents* ev) {
    (void)hipGetLastError();   // an earlier, unrelated failure is not ours to report
    set_keep_frac(b);
    EDKM_LAUNCH("k_init_zero", k_init_zero, dim3(T_WG, b.count), dim3(T_THREADS), b);
    EDKM_NPASS(PASS_HIST, "k_hist", k_hist, dim3(grid_np), dim3(NP_THREADS), b);
    EDKM_LAUNCH("k_hist_merge", k_hist_merge, dim3(W4 / MERGE_THREADS, merge_chunks(b), b.count),
                dim3(MERGE_THREADS), b);
    EDKM_LAUNCH("k_window", k_window, dim3(1, b.count), dim3(NP_THREADS), b);
    return hipSuccess;
}

hipError_t launch_forward(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                          const PassEvents* ev) {
    (void)hipGetLastError();
    set_keep_frac(b);
    EDKM_DISPATCH_K(b.m[0].k, forward_k, b, grid_np, max_t, s, where, ev);
}

hipError_t launch_backward(BatchArgs& b, uint32_t grid_np, int max_t, hipStream_t s, const char** where,
                           const PassEvents* ev) {
    (void)hipGetLastError();
    set_keep_frac(b);
    EDKM_DISPATCH_K(b.m[0].k, backward_k, b, grid_np, max_t, s, where, ev);
}

hipError_t launch_palettize(BatchArgs& b, uint32_t grid_np, hipStream_t s, const char** where,
                            const PassEvents* ev) {
    (void)hipGetLastError();
    EDKM_LAUNCH("k_pal_table", k_pal_table, dim3(NKEYS / 256, b.count), dim3(256), b);
    const dim3 grid(grid_np);
    switch (b.m[0].k) {
    case 2: EDKM_NPASS(PASS_PALETTIZE, "k_palettize", k_palettize<1>, grid, dim3(1024), b); break;
    case 4: EDKM_NPASS(PASS_PALETTIZE, "k_palettize", k_palettize<2>, grid, dim3(1024), b); break;
    case 8: EDKM_NPASS(PASS_PALETTIZE, "k_palettize", k_palettize<3>, grid, dim3(1024), b); break;
    case 16: EDKM_NPASS(PASS_PALETTIZE, "k_palettize", k_palettize<4>, grid, dim3(1024), b); break;
    default: return hipErrorInvalidValue;
    }
    return hipSuccess;
}

hipError_t launch_unique_inverse(BatchArgs& b, uint32_t grid_np, bool inverse, hipStream_t s,
                                 const char** where, const PassEvents* ev) {
    (void)hipGetLastError();
    EDKM_LAUNCH("k_rank", k_rank, dim3(1, b.count), dim3(1024), b);
    if (inverse) EDKM_NPASS(PASS_INVERSE, "k_inverse", k_inverse, dim3(grid_np), dim3(NP_THREADS), b);
    return hipSuccess;
}

hipError_t launch_forward_dense(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                const PassEvents* ev) {
    (void)hipGetLastError();
    EDKM_DISPATCH_K(b.m[0].k, forward_dense_k, b, nwg, s, where, ev);
}

hipError_t launch_backward_dense(BatchArgs& b, uint32_t nwg, hipStream_t s, const char** where,
                                 const PassEvents* ev) {
    (void)hipGetLastError();
    EDKM_DISPATCH_K(b.m[0].k, backward_dense_k, b, nwg, s, where, ev);
}

static_assert(W4 % NP_THREADS == 0, "merge grid covers the window exactly");
static_assert(2 * W8 <= ROW4, "keyed-reduction rows fit the partial-row stride");
static_assert(2 * W4 + 64 <= 2 * W8 * 2, "keyed sum: the 32-bit window and its spare words fit the LDS array");
static_assert(MAGS == (NP_THREADS / 64) * 8 * 256, "window selection: 8 chunks of 256 magnitudes per wave");
static_assert(fin_mags(FMT_FP16) % 4 == 0 && fin_mags(FMT_BF16) % 4 == 0,
              "window selection: a lane's 4 magnitudes are all finite or all not");
static_assert(T_WG % 64 == 0, "table partial reduction: one lane per 64 workgroups");
static_assert(T_WG * T_THREADS * T_KPT == NKEYS, "table blocks cover every pattern");

}  // namespace edkm

#ifdef EDKM_BLOCK_STAMPS
extern "C" int edkm_stamps_reset(void) {
    edkm::g_stamp_seq = 0;
    void* q = nullptr;
    hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(edkm::stamp_ts));
    if (e == hipSuccess) e = hipMemset(q, 0, sizeof(edkm::stamp_ts));
    if (e == hipSuccess) e = hipDeviceSynchronize();
    return (int)e;
}
extern "C" int edkm_stamps_dump(unsigned long long* stamps, char* names) {
    if (hipDeviceSynchronize() != hipSuccess) return -1;
    if (hipMemcpyFromSymbol(stamps, HIP_SYMBOL(edkm::stamp_ts), sizeof(edkm::stamp_ts)) != hipSuccess) return -1;
    for (int i = 0; i < edkm::STAMP_LAUNCHES * 32; ++i) names[i] = (&edkm::g_stamp_names[0][0])[i];
    return edkm::g_stamp_seq;
}
extern "C" int edkm_stamps_clock_khz(void) {
    int dev = 0, r = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&r, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
    return r;
}
#endif
