// gfx950 kernels of the Sol-Attn forward pass.
//
// Pipeline of one forward (bf16 inputs):
//   1. pool_mean      Qbar_i = token mean of query block i           (Eq. block_proxy)
//   2. prep_kv        Kbar_j (f32 + f16 copy), Vbar_j (f16, correction layout) and the
//                     f16 transposed V used by the exact tiles
//   3. moments        mean and centred covariance of the routable pooled keys, f64 sums
//   4. tau            tau_i = mu_i + beta*sigma_i from the moments   (Eqs. threshold_routing,
//                                                                       threshold_stats_exact)
//   4b. order         sparse modes: order of each head's query blocks in the attention
//                     kernel's work queues (scheduling: blocks with similar selections share an L2)
//   5. routed_attn    persistent workgroups claim (b, h, query block) items from per-XCD
//                     queues; per block: route every key block on chip from f32 proxies, then
//                     one online-softmax pass over correction tiles (pooled keys, Section 3.2
//                     "Proxy-Score Reuse") and exact tiles (selected key blocks), with bf16
//                     MFMA for QK^T and f16 MFMA for PV
//   6. count_reduce   per-head number of selected routable pairs
//
// Tile math (wave64, v_mfma_f32_32x32x16_{bf16,f16}): each wave owns 32 query rows and
// computes the transposed score tile S^T = K Q^T (keys on MFMA rows, queries on lanes), so a
// query's softmax state lives in one lane pair (l, l+32).  The probabilities are fed straight
// from the accumulator registers as the B operand of O^T += V^T P^T; for that the transposed
// V tiles store each 16-key segment with its two middle 4-key groups swapped, which makes the
// 8 keys a lane contributes contiguous in LDS.
#include "sol_attn_internal.h"

#include <algorithm>
#include <cmath>
#include <type_traits>

namespace sol {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
// Lazy rescaling: the running max subtracted from the logits (log2 units) is only raised
// when a tile's max exceeds it by more than this, so probabilities stay <= 2^8 (f16-safe).
constexpr float kRescaleSlack = 8.0f;
constexpr float kLog2BlockK = 6.0f;   // log2(64): multiplicity of a full key block, log2 units

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
    return __builtin_bit_cast(uint16_t, (__bf16)x);
}

// l + p.x + p.y in f32, from the two f16 halves of p exactly as they are: two mixed-precision
// FMAs (v_fma_mix_f32, each half times 1.0 plus the sum), the form of the row sums that issues
// beside the PV MFMAs of the tile loop (the f16 dot product stalls the matrix pipe there).
__device__ __forceinline__ float add_f16x2(float l, f16x2 p) {
    asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %0, %1, 1.0, %0 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "+v"(l)
        : "v"(p));
    return l;
}

// Position p of a transposed V row holds key swap23(p): bits 2 and 3 exchanged.
__device__ __forceinline__ int swap23(int p) {
    return (p & ~12) | ((p & 8) >> 1) | ((p & 4) << 1);
}

template <typename T>
struct Elem;
template <>
struct Elem<uint16_t> {
    static constexpr int kPerChunk = 8;
    __device__ static void unpack(const u32x4& c, float* out) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[2 * e] = bf16_bits_to_f32(c[e] & 0xffffu);
            out[2 * e + 1] = bf16_bits_to_f32(c[e] >> 16);
        }
    }
};
template <>
struct Elem<float> {
    static constexpr int kPerChunk = 4;
    __device__ static void unpack(const u32x4& c, float* out) {
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = __uint_as_float(c[e]);
    }
};

// ---------------------------------------------------------------------------
// Block mean pooling.  grid (nblocks, BH), 256 threads.  Each thread sums 16-byte
// chunks of a fixed column group over a strided set of rows; row groups are then
// combined through LDS.  Only the block's valid rows are read.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void pool_mean_block(const T* __restrict__ x, float* __restrict__ mean, int N, int D,
                                                int blk, int nb, int j, int bh) {
    constexpr int EPC = Elem<T>::kPerChunk;
    __shared__ float red[256 * EPC];
    const int t = threadIdx.x;
    const int cpr = D / EPC;
    const int groups = 256 / cpr;
    const int cc = t % cpr, g = t / cpr;
    const int row0 = j * blk;
    const int n = min(blk, N - row0);
    const T* base = x + ((size_t)bh * N + row0) * D + cc * EPC;
    float acc[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
    for (int r = g; r < n; r += groups) {
        u32x4 c = *reinterpret_cast<const u32x4*>(base + (size_t)r * D);
        float f[EPC];
        Elem<T>::unpack(c, f);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] += f[e];
    }
#pragma unroll
    for (int e = 0; e < EPC; ++e) red[g * D + cc * EPC + e] = acc[e];
    __syncthreads();
    const float inv = 1.0f / (float)n;
    for (int c = t; c < D; c += 256) {
        float s = 0.f;
        for (int gg = 0; gg < groups; ++gg) s += red[gg * D + c];
        mean[((size_t)bh * nb + j) * D + c] = s * inv;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void pool_mean_kernel(const T* __restrict__ x, float* __restrict__ mean,
                                                        int N, int D, int blk, int nb) {
    pool_mean_block<T>(x, mean, N, D, blk, nb, blockIdx.x, blockIdx.y);
}

// ---------------------------------------------------------------------------
// K/V preparation for the bf16 forward.  grid (NJ, BH), 256 threads, one key block each.
//   vt     [BH][NK][D][64] f16: V^T tile by tile (each key block's transposed values are
//          one contiguous 16 KB run at d = 128), swap23 key order inside each 16-key
//          segment; rows past N are zero.
//   routing modes additionally:
//   kbar   [BH][NK][D] f32 means (routing proxies and moments)
//   kbarh  [BH][NC*64][D] f16 key means of routable blocks (gathered into correction tiles);
//          zero for forced and padding rows
//   vbarh  [BH][NC*64][D] f16 value means, same rows
// Blocks j >= NK exist only to zero the padding rows of the last correction tile.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void prep_kv_kernel(const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
                                                      float* __restrict__ kbar, _Float16* __restrict__ kbarh,
                                                      _Float16* __restrict__ vbarh, _Float16* __restrict__ vt,
                                                      int N, int NK, int NKr, int NC, int routing) {
    constexpr int CPR = D / 8;          // 16-byte chunks per row
    constexpr int GROUPS = 256 / CPR;   // row groups
    constexpr int VS = D + 2;           // f16 row stride of the staged V tile (odd word count)
    __shared__ _Float16 vtile[kBlockK * VS];
    __shared__ float red[GROUPS * D];
    const int j = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
    const int cc = t % CPR, g = t / CPR;

    if (j >= NK) {  // padding rows of the last correction tile
        for (int c = t; c < D; c += 256) {
            kbarh[((size_t)bh * NC * kChunk + j) * D + c] = (_Float16)0.f;
            vbarh[((size_t)bh * NC * kChunk + j) * D + c] = (_Float16)0.f;
        }
        return;
    }
    const int row0 = j * kBlockK;
    const int n = min(kBlockK, N - row0);
    const float inv = 1.0f / (float)n;
    constexpr int RPT = kBlockK / GROUPS;   // rows per thread (4 or 2)

    // All loads of the block are issued up front: the thread's rows of V and, in routing
    // modes, of K (rows past N read as zero).
    u32x4 vraw[RPT], kraw[RPT];
    {
        const uint16_t* vb = v + ((size_t)bh * N + row0) * D + cc * 8;
        const uint16_t* kb = k + ((size_t)bh * N + row0) * D + cc * 8;
#pragma unroll
        for (int u = 0; u < RPT; ++u) {
            const int r = g + u * GROUPS;
            vraw[u] = r < n ? *reinterpret_cast<const u32x4*>(vb + (size_t)r * D) : u32x4{0u, 0u, 0u, 0u};
            kraw[u] = (routing && r < n) ? *reinterpret_cast<const u32x4*>(kb + (size_t)r * D) : u32x4{0u, 0u, 0u, 0u};
        }
    }
    // ---- V: stage as f16 (exact for bf16 values inside the f16 range) and sum columns
    {
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
        for (int u = 0; u < RPT; ++u) {
            const int r = g + u * GROUPS;
            float f[8];
            Elem<uint16_t>::unpack(vraw[u], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                acc[e] += f[e];
                vtile[r * VS + cc * 8 + e] = (_Float16)f[e];
            }
        }
        if (routing) {
#pragma unroll
            for (int e = 0; e < 8; ++e) red[g * D + cc * 8 + e] = acc[e];
        }
    }
    __syncthreads();
    // transposed write: thread -> (d row, run of consecutive positions)
    {
        constexpr int TPR = 256 / D;             // threads per d row (2 or 4)
        constexpr int RUN = kBlockK / TPR;       // positions per thread (32 or 16)
        const int drow = t / TPR, p0 = (t % TPR) * RUN;
        _Float16* dst = vt + (((size_t)bh * NK + j) * D + drow) * kBlockK + p0;
#pragma unroll
        for (int u = 0; u < RUN; u += 8) {
            f16x8 pk;
#pragma unroll
            for (int e = 0; e < 8; ++e) pk[e] = vtile[swap23(p0 + u + e) * VS + drow];
            *reinterpret_cast<f16x8*>(dst + u) = pk;
        }
    }
    if (!routing) return;
    if (t < D && j < NC * kChunk) {
        float s = 0.f;
        for (int gg = 0; gg < GROUPS; ++gg) s += red[gg * D + t];
        const bool routable = j < NKr;
        vbarh[((size_t)bh * NC * kChunk + j) * D + t] = routable ? (_Float16)(s * inv) : (_Float16)0.f;
    }
    __syncthreads();
    // ---- K: column means
    {
        float acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.f;
#pragma unroll
        for (int u = 0; u < RPT; ++u) {
            float f[8];
            Elem<uint16_t>::unpack(kraw[u], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] += f[e];
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) red[g * D + cc * 8 + e] = acc[e];
    }
    __syncthreads();
    if (t < D) {
        float s = 0.f;
        for (int gg = 0; gg < GROUPS; ++gg) s += red[gg * D + t];
        const float m = s * inv;
        kbar[((size_t)bh * NK + j) * D + t] = m;
        if (j < NC * kChunk)
            kbarh[((size_t)bh * NC * kChunk + j) * D + t] = j < NKr ? (_Float16)m : (_Float16)0.f;
    }
}

// ---------------------------------------------------------------------------
// Moments of the routable pooled keys (Eq. threshold_stats_exact, centred form), in two
// kernels.  moments_partial_kernel: grid (mom_splits(BH, NKr), BH), 256 threads; split s accumulates,
// in f64, S1 = sum_j x_j and S2 = sum_j x_j^T x_j over its share of the key blocks, with
// x_j = Kbar_j - Kbar_0 (a shift that keeps the second moment well conditioned).
// moments_final_kernel: grid (D*D/256, BH), sums the splits and writes mu_K = Kbar_0 + S1/n
// and C_K = S2/n - (S1/n)^T (S1/n) in f32, 256 entries of C_K per workgroup.
// ---------------------------------------------------------------------------
// Splits per head: as many as fill one round of the device's resident workgroups (two per CU
// at this kernel's register use), at most 32, and at least 32 pooled keys each (a split
// writes a d x d f64 partial, which the final kernel reads back).
constexpr int kMomMaxSplit = 32;
int mom_splits(int BH, int NKr) {
    return std::max(1, std::min({kMomMaxSplit, 512 / std::max(BH, 1), (NKr + 31) / 32}));
}

// Device lambdas of the attention kernel are always inlined: a call would move the register
// tile state through memory.
#define SOL_INLINE __attribute__((always_inline))

template <int D>
__device__ __forceinline__ void moments_partial_block(const float* __restrict__ kbar, double* __restrict__ part, int NK,
                                                      int NKr, int sp, int bh, int nsplit) {
    constexpr int SLAB = 32;
    constexpr int TS = D + 4;                  // f32 row stride of the staged slab
    constexpr int RB = D / 16;                 // 16x16 thread grid, RB x RB entries each
    __shared__ float x[SLAB * TS];
    __shared__ float k0[D];
    const int t = threadIdx.x;
    const float* kb = kbar + (size_t)bh * NK * D;
    const int j0 = (int)((long long)NKr * sp / nsplit), j1 = (int)((long long)NKr * (sp + 1) / nsplit);
    for (int c = t; c < D; c += 256) k0[c] = kb[c];
    __syncthreads();
    const int r0 = (t / 16) * RB, c0 = (t % 16) * RB;
    double s2[RB][RB];
    double s1 = 0.0;
#pragma unroll
    for (int u = 0; u < RB; ++u)
#pragma unroll
        for (int v = 0; v < RB; ++v) s2[u][v] = 0.0;
    for (int jb = j0; jb < j1; jb += SLAB) {
        const int rows = min(SLAB, j1 - jb);
        for (int e = t; e < rows * D; e += 256) x[(e / D) * TS + e % D] = kb[(size_t)(jb + e / D) * D + e % D] - k0[e % D];
        __syncthreads();
        for (int jj = 0; jj < rows; ++jj) {
            double xr[RB], xc[RB];
#pragma unroll
            for (int u = 0; u < RB; ++u) {
                xr[u] = x[jj * TS + r0 + u];
                xc[u] = x[jj * TS + c0 + u];
            }
#pragma unroll
            for (int u = 0; u < RB; ++u)
#pragma unroll
                for (int v = 0; v < RB; ++v) s2[u][v] = fma(xr[u], xc[v], s2[u][v]);
            if (t < D) s1 += (double)x[jj * TS + t];
        }
        __syncthreads();
    }
    double* out = part + ((size_t)bh * nsplit + sp) * (D * D + D);
#pragma unroll
    for (int u = 0; u < RB; ++u)
#pragma unroll
        for (int v = 0; v < RB; ++v) out[(r0 + u) * D + c0 + v] = s2[u][v];
    if (t < D) out[D * D + t] = s1;
}

template <int D>
__global__ __launch_bounds__(256) void moments_partial_kernel(const float* __restrict__ kbar, double* __restrict__ part,
                                                              int NK, int NKr, int nsplit) {
    moments_partial_block<D>(kbar, part, NK, NKr, blockIdx.x, blockIdx.y, nsplit);
}


template <int D>
__global__ __launch_bounds__(256) void moments_final_kernel(const float* __restrict__ kbar, const double* __restrict__ part,
                                                            float* __restrict__ muk, float* __restrict__ cov, int NK,
                                                            int NKr, int nsplit) {
    __shared__ double m[D];
    const int chunk = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
    const double* pp = part + (size_t)bh * nsplit * (D * D + D);
    const double inv = 1.0 / (double)NKr;
    for (int c = t; c < D; c += 256) {
        double s = 0.0;
        for (int sp = 0; sp < nsplit; ++sp) s += pp[(size_t)sp * (D * D + D) + D * D + c];
        m[c] = s * inv;
        if (chunk == 0) muk[(size_t)bh * D + c] = (float)((double)kbar[(size_t)bh * NK * D + c] + m[c]);
    }
    __syncthreads();
    const int e = chunk * 256 + t;
    if (e < D * D) {
        double s = 0.0;
        for (int sp = 0; sp < nsplit; ++sp) s += pp[(size_t)sp * (D * D + D) + e];
        cov[(size_t)bh * D * D + e] = (float)(s * inv - m[e / D] * m[e % D]);
    }
}

// ---------------------------------------------------------------------------
// Thresholds (Eq. threshold_routing with Eq. threshold_stats_exact, or with the diagonal
// estimator of the Appendix, Eq. appendix_diagonal_threshold, when DIAG).  grid (ceil(NQ/16), BH),
// 256 threads in 256/D groups of D.  Thread (g, r) holds column r of C_K (= row r, C_K is
// symmetric) in registers and, for the group's query blocks i, forms y_r = (C_K Qbar_i^T)_r
// from the staged Qbar rows (broadcast LDS reads); the D products Qbar_ir y_r and
// Qbar_ir mu_r are summed per wave, and the wave partials per query block give
// Qbar_i C_K Qbar_i^T and Qbar_i mu_K^T.
// ---------------------------------------------------------------------------
template <int D, bool DIAG>
__global__ __launch_bounds__(256) void tau_kernel(const float* __restrict__ qbar, const float* __restrict__ muk,
                                                  const float* __restrict__ cov, float* __restrict__ tau,
                                                  float* __restrict__ mu_out, float* __restrict__ sigma_out,
                                                  int NQ, float beta, float scale) {
    constexpr int QPB = 16;
    constexpr int PAR = 256 / D;      // groups
    constexpr int WPG = D / 64;       // waves per group
    __shared__ __attribute__((aligned(16))) float qs[QPB * D];
    __shared__ float red[QPB][WPG][2];
    const int bh = blockIdx.y, i0 = blockIdx.x * QPB, t = threadIdx.x;
    const int nq = min(QPB, NQ - i0);
    const int g = t / D, r = t % D, wv = r / 64, lane = t & 63;
    float ccol[DIAG ? 1 : D];
    if constexpr (DIAG) {
        ccol[0] = cov[((size_t)bh * D + r) * D + r];   // v_K[r], the diagonal of C_K
    } else {
#pragma unroll
        for (int c = 0; c < D; ++c) ccol[c] = cov[((size_t)bh * D + c) * D + r];
    }
    const float mkr = muk[(size_t)bh * D + r];
    for (int e = t; e < nq * D; e += 256) qs[e] = qbar[((size_t)bh * NQ + i0) * D + e];
    __syncthreads();
    for (int qq = g; qq < nq; qq += PAR) {
        const float* qrow = qs + qq * D;
        float y;
        if constexpr (DIAG) {
            y = ccol[0] * qrow[r];   // (diag(v_K) Qbar_i^T)_r
        } else {
            float y0 = 0.f, y1 = 0.f;
#pragma unroll
            for (int c = 0; c < D; c += 4) {
                const f32x4 qv = *reinterpret_cast<const f32x4*>(qrow + c);
                y0 = fmaf(ccol[c], qv[0], y0);
                y1 = fmaf(ccol[c + 1], qv[1], y1);
                y0 = fmaf(ccol[c + 2], qv[2], y0);
                y1 = fmaf(ccol[c + 3], qv[3], y1);
            }
            y = y0 + y1;
        }
        float w = qrow[r] * y;
        float m = qrow[r] * mkr;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            w += __shfl_xor(w, off);
            m += __shfl_xor(m, off);
        }
        if (lane == 0) {
            red[qq][wv][0] = w;
            red[qq][wv][1] = m;
        }
    }
    __syncthreads();
    if (t < nq) {
        float ws = 0.f, ms = 0.f;
#pragma unroll
        for (int u = 0; u < WPG; ++u) {
            ws += red[t][u][0];
            ms += red[t][u][1];
        }
        const float mu = scale * ms;
        const float sigma = scale * sqrtf(fmaxf(ws, 0.f));
        float th;
        if (beta == kNegInf) th = kNegInf;
        else if (beta == -kNegInf) th = -kNegInf;
        else th = mu + beta * sigma;
        const size_t o = (size_t)bh * NQ + i0 + t;
        tau[o] = th;
        if (mu_out) mu_out[o] = mu;
        if (sigma_out) sigma_out[o] = sigma;
    }
}

// ---------------------------------------------------------------------------
// Routing prologue shared by both attention kernels: the f32 proxy of every routable key
// block (pooled query . pooled key, scaled) against the row threshold (strict >) gives its
// selection bit for query block qi in selw (LDS); then two lists (LDS, 16-bit):
//   list[0, ucap)   the unselected routable blocks in increasing j (sparse mode): the slots
//                   of the correction tiles, 64 per tile, the last tile padded with block 0
//                   (ucap = 64 * the chunks of routable blocks);
//   list[ucap, ...) the exact tiles: selected routable blocks in increasing j, then the
//                   forced blocks.
// The online softmax is order independent, so running the correction tiles first changes
// only the floating-point summation order.  Returns the number of exact tiles; *nuns
// receives the number of unselected routable blocks and *nsel of selected ones.
//
// The routable blocks are [0, nr) and the forced ones [nr, ne): without a causal mask
// nr = NKr and ne = NK (the forced tail).  With a causal mask (CAUSAL) [0, nr) are the key
// blocks every row of the query block sees and [nr, ne) those only some rows see; the row
// statistics then cover [0, nr) only and are taken here, from the proxies themselves: the
// proxies go to LDS (prox, nr floats), their mean and population deviation give
// tau_i = mu_i + beta sigma_i, and the selection bits follow.  (Prefix moments of the pooled
// keys would need a d x d matrix per query block.)
// ---------------------------------------------------------------------------

// Sum over the workgroup; every thread gets the total.  scratch: NT/64 floats.
template <int NT>
__device__ float block_sum(float v, float* scratch) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) tot += scratch[w];
    __syncthreads();
    return tot;
}

template <int NT>
__device__ int block_scan_incl(int v, int* scratch, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int NW = NT / 64;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(v, off);
        if (lane >= off) v += y;
    }
    if (lane == 63) scratch[wave] = v;
    __syncthreads();
    int pre = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const int s = scratch[w];
        if (w < wave) pre += s;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return v + pre;
}

// ---------------------------------------------------------------------------
// Query-block order of the sparse kernels (scheduling only).
// The workgroups resident on one XCD share its L2, and a key block's tiles are served from L2
// only if the workgroups that select it read them close together in time.  Whether two query
// blocks select alike depends on their pooled queries as seen by the pooled keys: row i keeps
// key block j iff Qbar_i (Kbar_j - mu_K) exceeds beta sigma_i / s, so only the direction of
// Qbar_i in the space the pooled keys span matters.  The blocks of each head are therefore
// ordered along a Hilbert curve over (Qbar_i u1, Qbar_i u2) / sigma_i, with u1 and u2 the two
// leading eigenvectors of C_K (power iteration from fixed start vectors), and the sparse kernel
// hands consecutive blocks of that order to the same XCD.  Each query block is still computed
// by one workgroup exactly as in the identity order: the order decides which blocks run
// together, never a result.  Heads with more than kOrderMaxNQ query blocks keep the identity.
// ---------------------------------------------------------------------------
constexpr int kOrderMaxNQ = 4096;
constexpr int kOrderGrid = 256;   // Hilbert curve over a 256 x 256 grid: 16-bit indices

__device__ __forceinline__ uint32_t hilbert_index(uint32_t x, uint32_t y) {
    uint32_t d = 0;
    for (uint32_t s = kOrderGrid / 2; s > 0; s >>= 1) {
        const uint32_t rx = (x & s) ? 1u : 0u, ry = (y & s) ? 1u : 0u;
        d += s * s * ((3u * rx) ^ ry);
        if (ry == 0u) {   // rotate the quadrant
            if (rx == 1u) {
                x = kOrderGrid - 1 - x;
                y = kOrderGrid - 1 - y;
            }
            const uint32_t tmp = x;
            x = y;
            y = tmp;
        }
    }
    return d;
}

template <int NT>
__device__ float2 block_sum2(float x, float y, float2* scratch) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        x += __shfl_xor(x, off);
        y += __shfl_xor(y, off);
    }
    if (lane == 0) scratch[wave] = make_float2(x, y);
    __syncthreads();
    float2 tot = make_float2(0.f, 0.f);
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        tot.x += scratch[w].x;
        tot.y += scratch[w].y;
    }
    __syncthreads();
    return tot;
}

// KPT: query blocks ranked per thread, a power of two with 256 * KPT >= NQ (the launch picks the
// smallest), so that the rank loop runs no empty slots.
template <int D, int KPT>
__global__ __launch_bounds__(256) void order_kernel(const float* __restrict__ qbar, const float* __restrict__ cov,
                                                    const float* __restrict__ sigma, uint16_t* __restrict__ order,
                                                    int NQ) {
    constexpr int NT = 256;
    constexpr int ITERS = 4;         // power iterations per eigenvector: an offline study of the synthetic
                                     // workloads found the order as good as with 12
    __shared__ float u[2][D];
    __shared__ float vb[D];
    __shared__ float2 scratch2[NT / 64];
    __shared__ float red4[NT / 64][4];
    __shared__ float pa[kOrderMaxNQ], pb[kOrderMaxNQ];
    __shared__ __attribute__((aligned(16))) uint32_t keys[kOrderMaxNQ];
    const int bh = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
    uint16_t* ord = order + (size_t)bh * NQ;
    if (NQ > kOrderMaxNQ || NQ > NT * KPT) {
        for (int i = t; i < NQ; i += NT) ord[i] = (uint16_t)i;
        return;
    }
    // power iteration: u1, then u2 kept orthogonal to u1.  C_K is symmetric, so thread r < D
    // holds column r (= row r) in registers and forms (C v)_r from the vector in LDS.
    float ccol[D];
    if (t < D) {
#pragma unroll
        for (int c = 0; c < D; ++c) ccol[c] = cov[((size_t)bh * D + c) * D + t];
    }
    for (int e = 0; e < 2; ++e) {
        if (t < D) vb[t] = (float)((((uint32_t)t + 1u + 977u * (uint32_t)e) * 2654435761u) >> 22) / 1024.f - 0.5f;
        __syncthreads();
        for (int it = 0; it < ITERS; ++it) {
            float w = 0.f;
            if (t < D) {
                float w4[4] = {0.f, 0.f, 0.f, 0.f};   // four short chains
#pragma unroll
                for (int c = 0; c < D; ++c) w4[c & 3] = fmaf(ccol[c], vb[c], w4[c & 3]);
                w = (w4[0] + w4[1]) + (w4[2] + w4[3]);
            }
            // one reduction for |w|^2 and u1.w: |w - (u1.w) u1|^2 = |w|^2 - (u1.w)^2 for unit u1
            const float2 r = block_sum2<NT>(t < D ? w * w : 0.f, (t < D && e == 1) ? w * u[0][t] : 0.f, scratch2);
            if (e == 1 && t < D) w -= r.y * u[0][t];
            const float nrm = sqrtf(fmaxf(r.x - (e == 1 ? r.y * r.y : 0.f), 0.f));
            if (t < D) vb[t] = nrm > 0.f ? w / nrm : 0.f;
            __syncthreads();
        }
        if (t < D) u[e][t] = vb[t];
        __syncthreads();
    }
    // projections (Qbar_i u1, Qbar_i u2) / sigma_i, one thread per row (16-byte row reads, no
    // cross-lane reductions); u1 and u2 are broadcast from LDS
    for (int i = t; i < NQ; i += NT) {
        const f32x4* qr = reinterpret_cast<const f32x4*>(qbar + ((size_t)bh * NQ + i) * D);
        float a4[4] = {0.f, 0.f, 0.f, 0.f}, b4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const f32x4 qv = qr[c4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                a4[e] = fmaf(qv[e], u[0][4 * c4 + e], a4[e]);
                b4[e] = fmaf(qv[e], u[1][4 * c4 + e], b4[e]);
            }
        }
        const float sg = sigma[(size_t)bh * NQ + i];
        const float inv = sg > 0.f ? 1.f / sg : 1.f;
        pa[i] = ((a4[0] + a4[1]) + (a4[2] + a4[3])) * inv;
        pb[i] = ((b4[0] + b4[1]) + (b4[2] + b4[3])) * inv;
    }
    __syncthreads();
    // bounding box of the projections: one reduction of four maxima
    float m4[4] = {-__builtin_huge_valf(), -__builtin_huge_valf(), -__builtin_huge_valf(), -__builtin_huge_valf()};
    for (int i = t; i < NQ; i += NT) {
        m4[0] = fmaxf(m4[0], pa[i]);
        m4[1] = fmaxf(m4[1], -pa[i]);
        m4[2] = fmaxf(m4[2], pb[i]);
        m4[3] = fmaxf(m4[3], -pb[i]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) m4[q] = fmaxf(m4[q], __shfl_xor(m4[q], off));
    }
    if (lane == 0)
#pragma unroll
        for (int q = 0; q < 4; ++q) red4[wave][q] = m4[q];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        m4[q] = red4[0][q];
#pragma unroll
        for (int w = 1; w < NT / 64; ++w) m4[q] = fmaxf(m4[q], red4[w][q]);
    }
    const float amax = m4[0], amin = -m4[1], bmax = m4[2], bmin = -m4[3];
    const float ascl = amax > amin ? (float)(kOrderGrid - 1) / (amax - amin) : 0.f;
    const float bscl = bmax > bmin ? (float)(kOrderGrid - 1) / (bmax - bmin) : 0.f;
    for (int i = t; i < NQ; i += NT) {
        const uint32_t gx = (uint32_t)min(kOrderGrid - 1, max(0, (int)((pa[i] - amin) * ascl + 0.5f)));
        const uint32_t gy = (uint32_t)min(kOrderGrid - 1, max(0, (int)((pb[i] - bmin) * bscl + 0.5f)));
        keys[i] = (hilbert_index(gx, gy) << 16) | (uint32_t)i;   // distinct: the block index is in the low bits
    }
    for (int i = NQ + t; i < ((NQ + 3) & ~3); i += NT) keys[i] = 0xffffffffu;   // pad to whole 16-byte reads
    __syncthreads();
    // rank sort: block i goes to position |{j : key_j < key_i}|.  Each thread ranks all of its
    // keys (at most KPT) in one pass over the keys, read four at a time.
    static_assert(NT * KPT <= kOrderMaxNQ, "rank slots exceed the key buffer");
    uint32_t mine[KPT];
    int rank[KPT];
#pragma unroll
    for (int r = 0; r < KPT; ++r) {
        const int i = t + NT * r;
        mine[r] = i < NQ ? keys[i] : 0u;
        rank[r] = 0;
    }
    const int nmine = (NQ - t + NT - 1) / NT;   // keys this thread owns (wave-divergent only at the edge)
    const uint4* k4 = reinterpret_cast<const uint4*>(keys);
    for (int j4 = 0; j4 < (NQ + 3) / 4; ++j4) {
        const uint4 kj = k4[j4];
#pragma unroll
        for (int r = 0; r < KPT; ++r) {
            if (r < nmine)
                rank[r] += (kj.x < mine[r] ? 1 : 0) + (kj.y < mine[r] ? 1 : 0) + (kj.z < mine[r] ? 1 : 0) +
                           (kj.w < mine[r] ? 1 : 0);
        }
    }
#pragma unroll
    for (int r = 0; r < KPT; ++r)
        if (r < nmine) ord[rank[r]] = (uint16_t)(t + NT * r);
}

template <int D, int NT, int MODE, bool CAUSAL = false>
__device__ int route_and_list(const float* __restrict__ qbar_i, const float* __restrict__ kbar_h, float tau_i,
                              float beta, float scale, int NKr, int nr, int ne, int MW, float* prox, uint32_t* selw,
                              uint16_t* list, int ucap, int* scan_scratch, int* wpre, int* nuns, int* nsel) {
    const int NC = (nr + kChunk - 1) / kChunk;   // chunks of routable blocks
    constexpr int CPR = D / 4;              // 16-byte chunks per f32 pooled-key row
    constexpr int TPK = NT / kChunk;        // threads per pooled key (1, 2 or 4)
    constexpr int CPT = CPR / TPK;          // 16-byte chunks of a row per thread
    constexpr int KPWV = 64 / TPK;          // pooled keys per wave (64, 32 or 16)
    static_assert(NT % kChunk == 0 && TPK <= 4, "routing expects 64..256 threads");
    int tid_ = threadIdx.x;
    asm volatile("" : "+v"(tid_));   // per-lane values formed here, not hoisted out of a block loop
    const int tid = tid_, lane = tid & 63, wave = tid >> 6;
    const int jl = tid / TPK, seg = tid % TPK;
    // Each thread streams its share (chunks seg, seg+TPK, ...) of one pooled-key row per group
    // of 64 keys straight from L2 into registers, up to three groups in flight; the pooled
    // query stays in registers.  No LDS staging and no barrier until all proxies are decided.
    f32x4 qv[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) qv[i] = *reinterpret_cast<const f32x4*>(qbar_i + 4 * (seg + TPK * i));
    auto load = [&](int c, f32x4 (&kv)[CPT]) SOL_INLINE {
        const float* rp = kbar_h + (size_t)min(c * kChunk + jl, nr - 1) * D;
#pragma unroll
        for (int i = 0; i < CPT; ++i) kv[i] = *reinterpret_cast<const f32x4*>(rp + 4 * (seg + TPK * i));
    };
    auto decide = [&](int c, const f32x4 (&kv)[CPT]) SOL_INLINE {
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            a0 = fmaf(qv[i][0], kv[i][0], a0);
            a1 = fmaf(qv[i][1], kv[i][1], a1);
            a2 = fmaf(qv[i][2], kv[i][2], a2);
            a3 = fmaf(qv[i][3], kv[i][3], a3);
        }
        float dot = (a0 + a1) + (a2 + a3);
        // the TPK lanes of a key are consecutive lanes of one quad: reduce with quad
        // permutations (DPP), which stay in the VALU instead of going through the LDS crossbar
        if constexpr (TPK >= 2)
            dot += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(dot), 0xB1, 0xF, 0xF, false));
        if constexpr (TPK >= 4)
            dot += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(dot), 0x4E, 0xF, 0xF, false));
        const int j = c * kChunk + jl;
        if constexpr (CAUSAL) {
            if (seg == 0 && j < nr) prox[j] = scale * dot;
            return;
        }
        const bool sel = j < nr && scale * dot > tau_i;
        const uint64_t bal = __ballot(sel);
        // every TPK-th ballot bit (all lanes of a key agree): compress them into KPWV bits
        uint64_t bits = bal;
        if constexpr (TPK == 4) {
            bits &= 0x1111111111111111ull;
            bits = (bits | (bits >> 3)) & 0x0303030303030303ull;
            bits = (bits | (bits >> 6)) & 0x000F000F000F000Full;
            bits = (bits | (bits >> 12)) & 0x000000FF000000FFull;
            bits = (bits | (bits >> 24)) & 0xFFFFull;
        } else if constexpr (TPK == 2) {
            bits &= 0x5555555555555555ull;
            bits = (bits | (bits >> 1)) & 0x3333333333333333ull;
            bits = (bits | (bits >> 2)) & 0x0F0F0F0F0F0F0F0Full;
            bits = (bits | (bits >> 4)) & 0x00FF00FF00FF00FFull;
            bits = (bits | (bits >> 8)) & 0x0000FFFF0000FFFFull;
            bits = (bits | (bits >> 16)) & 0xFFFFFFFFull;
        }
        if (lane == 0) {
            const int bit0 = c * kChunk + wave * KPWV;
            if constexpr (KPWV == 64) {
                selw[bit0 >> 5] = (uint32_t)bits;
                if ((bit0 >> 5) + 1 < MW) selw[(bit0 >> 5) + 1] = (uint32_t)(bits >> 32);
            } else if constexpr (KPWV == 32) {
                if ((bit0 >> 5) < MW) selw[bit0 >> 5] = (uint32_t)bits;
            } else {
                if ((bit0 >> 5) < MW) reinterpret_cast<uint16_t*>(selw)[bit0 >> 4] = (uint16_t)bits;
            }
        }
    };
    // ring of NB groups in flight (fewer when a thread's share of a row is large)
    constexpr int NB = CPT <= 8 ? 3 : (CPT <= 16 ? 2 : 1);
    f32x4 kb[NB][CPT];
    // Loads of rows past the routable keys are clamped to the last one, so they are always
    // issued: with no conditional load in the steady-state loop the compiler's wait counts
    // cover exactly the group being decided and the other NB - 1 groups stay in flight.
#pragma unroll
    for (int b = 0; b < NB; ++b) load(b, kb[b]);
    int c = 0;
    for (; c + 2 * NB <= NC; c += NB) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            decide(c + b, kb[b]);
            load(c + b + NB, kb[b]);
        }
    }
    // tail: fewer than 2 NB groups left (all of them when NC < NB)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (c + b < NC) decide(c + b, kb[b]);
        if (c + b + NB < NC) load(c + b + NB, kb[b]);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
        if (c + NB + b < NC) decide(c + NB + b, kb[b]);
    __syncthreads();
    if constexpr (CAUSAL) {
        // row statistics over the routable prefix, then the selection bits of every word
        float* fscratch = reinterpret_cast<float*>(scan_scratch);
        float th = -kNegInf;
        if (nr > 0) {
            float acc = 0.f;
            for (int j = tid; j < nr; j += NT) acc += prox[j];
            const float mu = block_sum<NT>(acc, fscratch) / (float)nr;
            acc = 0.f;
            for (int j = tid; j < nr; j += NT) {
                const float dv = prox[j] - mu;
                acc = fmaf(dv, dv, acc);
            }
            const float sigma = sqrtf(block_sum<NT>(acc, fscratch) / (float)nr);
            if (beta == kNegInf) th = kNegInf;
            else if (beta == -kNegInf) th = -kNegInf;
            else th = mu + beta * sigma;
        }
        for (int w = tid; w < MW; w += NT) {
            uint32_t bits = 0u;
            for (int b = 0; b < 32; ++b) {
                const int j = 32 * w + b;
                if (j < nr && prox[j] > th) bits |= 1u << b;
            }
            selw[w] = bits;
        }
        __syncthreads();
    }
    uint16_t* ulist = list;          // unselected routable blocks, increasing j (sparse mode), padded
    uint16_t* elist = list + ucap;   // selected routable blocks, increasing j, then the forced ones
    // Both lists in one pass with a thread per block: a scan of the words' popcounts gives the
    // selected blocks before each word, a popcount within the word those before block j; j is
    // then selected block number `before` and, if not selected, unselected block j - before.
    const int MWr = (nr + 31) >> 5;  // words holding routable bits (bits past nr are zero)
    int n_sel = 0;
    for (int w0 = 0; w0 < MWr; w0 += NT) {
        const int w = w0 + tid;
        const int cnt = w < MWr ? __popc(selw[w]) : 0;
        int tot;
        const int incl = block_scan_incl<NT>(cnt, scan_scratch, &tot);
        if (w < MWr) wpre[w] = n_sel + incl - cnt;
        n_sel += tot;
    }
    __syncthreads();
    for (int j = tid; j < nr; j += NT) {
        const uint32_t word = selw[j >> 5];
        const int b = j & 31;
        const int before = wpre[j >> 5] + __popc(word & ((1u << b) - 1u));
        if ((word >> b) & 1u) elist[before] = (uint16_t)j;
        else if (MODE == kSparse) ulist[j - before] = (uint16_t)j;
    }
    const int n_uns = MODE == kSparse ? nr - n_sel : 0;
    // pad the last correction tile's slots with block 0 (their scores are masked), so that the
    // tile copies read the list without bounds checks
    if (MODE == kSparse)
        for (int u = n_uns + tid; u < ((n_uns + kChunk - 1) / kChunk) * kChunk; u += NT) ulist[u] = 0;
    for (int j = nr + tid; j < ne; j += NT) elist[n_sel + (j - nr)] = (uint16_t)j;
    __syncthreads();
    *nuns = n_uns;
    *nsel = n_sel;
    return n_sel + (ne - nr);
}

// ---------------------------------------------------------------------------
// Fused routed attention, bf16 inputs.
// ---------------------------------------------------------------------------
struct AttnArgs {
    const uint16_t* q;
    const uint16_t* k;
    const _Float16* vt;
    const float* qbar;
    const float* kbar;
    const _Float16* kbarh;
    const _Float16* vbarh;
    const float* tau;
    uint16_t* out;
    uint32_t* blkcount;
    uint32_t* mask_out;
    const uint16_t* order;        // [BH][NQ] query-block order (sparse modes), or null: identity
    uint32_t* queue;              // [8][32] per-XCD claim counters, zero at launch
    int resident;                 // workgroups per XCD in the persistent grid (grid / 8)
    int hlog;                     // log2 of the heads whose blocks are in the queues at once (no causal mask)
    int BH, N, NQ, NK, NKr, NC, MW, per_x;
    float scale, c_log2;
    float bias_full, bias_last;   // log2(n_j)/c_log2 for full blocks and for the last block
    int causal_g;                 // causal granule G (CAUSAL kernels): key s visible to query t iff s < lim(t)
    float beta;                   // standardised cutoff (CAUSAL kernels take tau_i on chip)
};

// Causal masks: query t sees the keys s < lim(t) = min((t / G + 1) G, N).  For query block qi
// of BQ rows, [0, nr) are the key blocks all its rows see and [nr, ne) those some rows see.
__device__ __forceinline__ int causal_lim(int t, int G, int N) { return min((t / G + 1) * G, N); }
template <int BQ>
__device__ __forceinline__ void causal_ranges(int qi, int G, int N, int NK, int& nr, int& ne) {
    const int lo = causal_lim(qi * BQ, G, N);
    const int hi = causal_lim(min((qi + 1) * BQ, N) - 1, G, N);
    nr = lo >= N ? NK : lo / kBlockK;
    ne = (hi + kBlockK - 1) / kBlockK;
}

// LDS tiles of the fused kernel, without padding.  gfx950 serves a ds_read_b128 16 lanes per
// cycle from 64 banks, so 16 consecutive MFMA rows reading the same 16-byte chunk column must
// land on 16 different bank groups.
//  * K tile (64 rows x D bf16, KCPR = D/8 chunks per row): for D = 128 chunk c of row r sits at
//    position r*16 + (c ^ (r mod 16)); for D = 64 rows pair into super-rows as below.
//  * V^T tile (D rows x 64 f16, 8 chunks per row): rows 2R and 2R+1 form a 16-chunk super-row R;
//    chunk c of row r is super-chunk C = c + 8*(r&1), stored at R*16 + (C ^ (R mod 16)).
// ksrc()/vsrc() invert the maps for the copy side: LDS chunk position -> (row, chunk).
template <int D>
struct TileLds {
    static constexpr int KCPR = D / 8;
    static constexpr int VCPR = kBlockK / 8;
    static constexpr int KBYTES = kBlockK * D * 2;
    static constexpr int VBYTES = D * kBlockK * 2;
    static constexpr int STAGE = KBYTES + VBYTES;
    // 16-chunk rows (D = 128): XOR with 4 row bits; 8-chunk rows (D = 64): super-rows as for V^T
    __device__ static int kpos(int r, int c) {
        if constexpr (KCPR == 16) return r * 16 + (c ^ (r & 15));
        const int R = r >> 1;
        return R * 16 + ((c + 8 * (r & 1)) ^ (R & 15));
    }
    __device__ static void ksrc(int p, int& r, int& c) {
        const int R = p >> 4;
        const int C = (p & 15) ^ (R & 15);
        if constexpr (KCPR == 16) {
            r = R;
            c = C;
        } else {
            r = 2 * R + (C >> 3);
            c = C & 7;
        }
    }
    __device__ static int vpos(int r, int c) {
        const int R = r >> 1;
        return R * 16 + ((c + 8 * (r & 1)) ^ (R & 15));
    }
    __device__ static void vsrc(int p, int& r, int& c) {
        const int R = p >> 4;
        const int C = (p & 15) ^ (R & 15);
        r = 2 * R + (C >> 3);
        c = C & 7;
    }
    // Correction tiles keep their value means row-major in the V region: slot s at s * 2D
    // bytes, chunk q of the row holding chunk q ^ rswz(s).  The correction PV reads it with
    // transposed loads, 32 lanes covering 4 consecutive slots x 4 consecutive chunks; rswz
    // puts those 16 chunks in distinct bank groups.
    static constexpr int RCPR = D / 8;
    __device__ static int rswz(int s) { return RCPR == 16 ? 4 * (s & 3) : 4 * ((s >> 1) & 1); }
    __device__ static void rsrc(int p, int& s, int& c) {
        s = p / RCPR;
        c = (p % RCPR) ^ rswz(s);
    }
};

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4* lds_s16x4_ptr;

// Transposed LDS read (ds_read_b64_tr_b16).  Within each group of 16 lanes, lane j supplies
// the address of 4 consecutive 16-bit values R_j; lane i receives R_{4e + i/4}[i % 4] for
// e = 0..3.  With lane j pointing at row j/4, columns 4*(j%4).., lane i gets column i of
// 4 consecutive rows.
__device__ __forceinline__ s16x4 lds_read_tr16(const char* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr)(p));
}

// Direct global->LDS copy of 16 bytes per lane (LDS bytes [dst + 16*lane, +16)), written as
// inline assembly so that the compiler's wait-count model does not track it: the exact-tile
// loop orders its copies with its own s_waitcnt/barrier pairs, and the compiler, which would
// otherwise treat every later LDS read as possibly aliasing an in-flight copy, is left free
// to schedule the operand reads.  dst must be wave-uniform (it goes to m0); the s_nop covers
// the one-wait-state hazard between an m0 write and an LDS DMA that reads it.
// The address is a wave-uniform base (scalar registers) plus a per-lane 32-bit byte offset,
// so no per-lane 64-bit address arithmetic is needed.
__device__ __forceinline__ void lds_copy16(const void* base, uint32_t off, lds_ptr_t dst) {
    const uint32_t m0 = (uint32_t)(uintptr_t)dst;
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(m0) : "memory");
}

// Key split: at d = 128 the LDS of a workgroup (two 32 KB tile stages) leaves room for two
// workgroups per CU, so a 64-row query block with one wave per 32 rows would run one wave per
// SIMD.  Instead its workgroup has four waves: wave w owns rows 32*(w%2).. and the key half
// w/2 (32 keys) of every tile, runs its own online softmax over those keys, and the two states
// of each row merge at the end.  That gives two waves per SIMD with half the MFMAs per wave.
template <int D, int BQ>
constexpr bool kAttnKeySplit = (D == 128 && BQ == 64);
template <int D, int BQ>
constexpr int kAttnThreads = kAttnKeySplit<D, BQ> ? 256 : BQ * 2;

// Every instantiation is register-budgeted for two waves per SIMD.
// One query block (b, h, qi) of the fused kernel; y is its position in its XCD's queue.
template <int D, int BQ, int MODE, bool CAUSAL>
__device__ __forceinline__ void attn_block(const AttnArgs& a, char* smem, const int bh, const int qi, const int y) {
    constexpr bool KSPLIT = kAttnKeySplit<D, BQ>;
    constexpr int NT = kAttnThreads<D, BQ>;   // 64 threads per 32 query rows (per key half)
    constexpr int NW = NT / 64;
    constexpr int NS = KSPLIT ? 1 : 2;       // 32-key score M-tiles per wave and tile
    constexpr int NPB = 2 * NS;              // 16-key P blocks per wave and tile
    using L = TileLds<D>;
    constexpr int KPW = L::KBYTES / 1024 / NW;   // direct-to-LDS wave loads per wave (K tile)
    constexpr int VPW = L::VBYTES / 1024 / NW;   // same for the V^T tile
    constexpr int NDT = D / 32;           // output M-tiles (d rows)
    constexpr int NKS = D / 16;           // k-steps of QK^T

    // The thread index is made opaque here so that the per-lane constants derived from it are
    // formed anew for every block rather than hoisted out of the block loop, where they would
    // stay live through it and push the tile loop past its register budget.
    int tid_ = threadIdx.x;
    asm volatile("" : "+v"(tid_));
    const int tid = tid_, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, kept in an SGPR
    const int r32 = lane & 31, hh = lane >> 5;
    const int rw = KSPLIT ? (wave & 1) : wave;   // 32-row slice of the query block
    const int kh = KSPLIT ? (wave >> 1) : 0;     // key half of every tile (key split only)
    const int kbase = 32 * kh;                   // first tile key of this wave's scores

    char* rest = smem + 2 * L::STAGE;
    int* scan_scratch = reinterpret_cast<int*>(rest);
    uint32_t* selw = reinterpret_cast<uint32_t*>(rest + 64);
    uint16_t* list = reinterpret_cast<uint16_t*>(rest + 64 + 4 * ((a.MW + 3) & ~3));
    int* wpre = reinterpret_cast<int*>(rest + ((64 + 4 * ((a.MW + 3) & ~3) + 2 * (a.NC * kChunk + a.NK) + 15) & ~15));
    // The causal prologue's per-row proxies: in the tile stages, which no copy fills before the
    // routing is done (the block loop's barrier ends every read of the previous block's tiles),
    // when they fit there; else after the word prefixes.
    float* prox = 4 * a.NKr <= 2 * L::STAGE ? reinterpret_cast<float*>(smem)
                                             : reinterpret_cast<float*>(wpre + ((a.MW + 3) & ~3));
    const uint16_t* ulist = list;            // correction slots (unselected routable blocks, padded)
    const uint16_t* elist = list + a.NC * kChunk;   // exact tiles

    int nr = a.NKr, ne = a.NK;               // routable blocks [0, nr), forced blocks [nr, ne)
    if constexpr (CAUSAL) causal_ranges<BQ>(qi, a.causal_g, a.N, a.NK, nr, ne);
    int ntiles, nsel, nuns = 0;
    if (MODE == kDense) {
        ntiles = ne;
        nsel = nr;
    } else {
        const float tau_i = CAUSAL ? 0.f : a.tau[(size_t)bh * a.NQ + qi];
        ntiles = route_and_list<D, NT, MODE, CAUSAL>(a.qbar + ((size_t)bh * a.NQ + qi) * D,
                                                     a.kbar + (size_t)bh * a.NK * D, tau_i, a.beta, a.scale, a.NKr,
                                                     nr, ne, a.MW, prox, selw, list, a.NC * kChunk, scan_scratch,
                                                     wpre, &nuns, &nsel);
        if (a.mask_out)
            for (int w = tid; w < a.MW; w += NT) a.mask_out[((size_t)bh * a.NQ + qi) * a.MW + w] = selw[w];
    }
    if (tid == 0) a.blkcount[(size_t)bh * a.NQ + qi] = (uint32_t)nsel;
    const int napx = MODE == kSparse ? (nuns + kChunk - 1) / kChunk : 0;   // correction tiles
    // slot of the ragged last key block among the correction slots (it can only be the last one)
    const int last_slot = (nuns > 0 && a.NKr == a.NK && ulist[max(nuns - 1, 0)] == a.NK - 1) ? nuns - 1 : -1;

    const int qrow = qi * BQ + rw * 32 + r32;
    const uint16_t* qrow_p = a.q + ((size_t)bh * a.N + min(qrow, a.N - 1)) * D + 8 * hh;
    const int qlim = CAUSAL ? causal_lim(qrow, a.causal_g, a.N) : a.N;   // this lane's query sees keys < qlim

    f32x16 o[NDT];
#pragma unroll
    for (int mt = 0; mt < NDT; ++mt) o[mt] = f32x16{};
    // Row sum of the probabilities in four partial sums, one per 16-key block of a tile, so
    // that the dot-product accumulations of a tile form four short dependency chains.
    float m_run = kNegInf, l_run[4] = {0.f, 0.f, 0.f, 0.f};

    // Start phase of the exact tiles (sparse modes, no causal mask).  A block walks its selected
    // key blocks in increasing order.  The first R blocks of an XCD's queue (R = the workgroups
    // of the persistent grid on one XCD, 64 at d = 128) start together at key block 0; later ones
    // start whenever a workgroup finishes, while the others are part-way through their lists,
    // so their tiles are no longer in L2 when the newcomer asks for them.  The block at queue
    // position y >= R therefore starts its walk at j0 = ((y - R) mod R) / R of the unselected
    // count and wraps round, which spreads the newcomers over the key range the way the running
    // blocks are spread.  With every block selected j0 = 0, so that case keeps dense mode's tile
    // order exactly.  The ragged last key block, when selected, stays the last tile (its tail
    // mask is applied after the loop).
    int k0 = 0, nrot = 0;
    if constexpr (MODE != kDense && !CAUSAL) {
        const bool ragged_last = nsel > 0 && a.NKr == a.NK && (a.N % kBlockK) != 0 && elist[nsel - 1] == a.NK - 1;
        nrot = nsel - (ragged_last ? 1 : 0);
        const int R = a.resident;
        const int j0 = y < R ? 0 : ((y - R) % R) * (a.NKr - nsel) / R;
        int lo = 0, hi = nrot;          // first position with elist[k] >= j0
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if ((int)elist[mid] < j0) lo = mid + 1;
            else hi = mid;
        }
        k0 = lo < nrot ? lo : 0;
        k0 = __builtin_amdgcn_readfirstlane(k0);
    }
    auto tile_code = [&](int n) -> int {
        if constexpr (MODE == kDense) return n;
        else {
            int k = n;
            if (n < nrot) {
                k = n + k0;
                if (k >= nrot) k -= nrot;
            }
            return (int)elist[k];
        }
    };
    // Global->LDS copies.  Each lane moves one 16-byte chunk per instruction; the per-lane
    // byte offsets inside a tile are fixed, so they are computed once here and each tile only
    // adds wave-uniform base pointers.  Rows past the end of the sequence (ragged last block)
    // are clamped to the last valid row: their scores are masked to -inf and their values
    // are zero in V^T.  Two-wave workgroups issue twice as many copies per wave and recompute
    // the offsets instead of holding them in registers.
    constexpr bool kKeepOff = NW >= 4;
    auto kofs_calc = [&](int u) SOL_INLINE -> uint32_t {
        int r, c;
        L::ksrc((wave * KPW + u) * 64 + lane, r, c);
        return (uint32_t)(r * D + c * 8) * 2u;
    };
    auto vofs_calc = [&](int u) SOL_INLINE -> uint32_t {
        int r, c;
        L::vsrc((wave * VPW + u) * 64 + lane, r, c);
        return (uint32_t)(r * kBlockK + c * 8) * 2u;
    };
    uint32_t koff[kKeepOff ? KPW : 1], voff[kKeepOff ? VPW : 1];
    if constexpr (kKeepOff) {
#pragma unroll
        for (int u = 0; u < KPW; ++u) koff[u] = kofs_calc(u);
#pragma unroll
        for (int u = 0; u < VPW; ++u) voff[u] = vofs_calc(u);
    }
    auto kofs = [&](int u) SOL_INLINE -> uint32_t {
        if constexpr (kKeepOff) return koff[u];
        else return kofs_calc(u);
    };
    auto vofs = [&](int u) SOL_INLINE -> uint32_t {
        if constexpr (kKeepOff) return voff[u];
        else return vofs_calc(u);
    };
    // Copies of correction tile c: the f16 pooled keys of its 64 slots (gathered rows; padding
    // slots past the unselected blocks copy row 0, their scores are masked) into stage `buf`'s
    // K region, K layout ...
    auto slot_row = [&](int c, int r) SOL_INLINE -> int {
        return ulist[c * kChunk + r];   // padding slots of the last tile hold block 0
    };
    const char* kbh_base = reinterpret_cast<const char*>(a.kbarh + (size_t)bh * a.NC * kChunk * D);
    const char* vbh_base = reinterpret_cast<const char*>(a.vbarh + (size_t)bh * a.NC * kChunk * D);
    auto issue_apx_k = [&](int c, int buf) SOL_INLINE {
        char* stage = smem + buf * L::STAGE;
        // all row lookups first, so that they are in flight together (each copy is ordered
        // after every memory access before it)
        uint32_t off[KPW];
#pragma unroll
        for (int u = 0; u < KPW; ++u) {
            int r, cc;
            if constexpr (L::KCPR == 16) {   // copy u covers rows 4(wave*KPW+u) .. +3, 16 lanes each
                r = 4 * (wave * KPW + u) + (lane >> 4);
                cc = (lane & 15) ^ (r & 15);
            } else {
                L::ksrc((wave * KPW + u) * 64 + lane, r, cc);
            }
            off[u] = (uint32_t)(slot_row(c, r) * D + cc * 8) * 2u;
        }
#pragma unroll
        for (int u = 0; u < KPW; ++u) lds_copy16(kbh_base, off[u], (lds_ptr_t)(stage + (wave * KPW + u) * 1024));
    };
    // ... and the f16 value means of the same rows into its V region, row-major (slot s at
    // s * 2D bytes, 16-byte chunk q of a row holding chunk q ^ rswz(s)), read back transposed
    // by the correction PV ...
    auto issue_apx_v = [&](int c, int buf) SOL_INLINE {
        char* stage = smem + buf * L::STAGE;
        constexpr int LPR = L::RCPR;                  // lanes per row of a copy
        const int cc = (lane % LPR) ^ L::rswz(lane / LPR);   // rswz depends on the row mod 4
        uint32_t off[VPW];
#pragma unroll
        for (int u = 0; u < VPW; ++u) {
            const int r = (64 / LPR) * (wave * VPW + u) + lane / LPR;
            off[u] = (uint32_t)(slot_row(c, r) * D + cc * 8) * 2u;
        }
#pragma unroll
        for (int u = 0; u < VPW; ++u)
            lds_copy16(vbh_base, off[u], (lds_ptr_t)(stage + L::KBYTES + (wave * VPW + u) * 1024));
    };
    // ... and of an exact tile: key block j into stage `buf`'s K region ...
    auto issue_exact_k = [&](int j, int buf) SOL_INLINE {
        j = __builtin_amdgcn_readfirstlane(j);   // the same block for every lane: scalar base address
        char* stage = smem + buf * L::STAGE;
        const char* kp = reinterpret_cast<const char*>(a.k + ((size_t)bh * a.N + (size_t)j * kBlockK) * D);
        const int nrows = a.N - j * kBlockK;
        if (nrows >= kBlockK) {
#pragma unroll
            for (int u = 0; u < KPW; ++u)
                lds_copy16(kp, kofs(u), (lds_ptr_t)(stage + (wave * KPW + u) * 1024));
        } else {
#pragma unroll
            for (int u = 0; u < KPW; ++u) {
                int r, c;
                L::ksrc((wave * KPW + u) * 64 + lane, r, c);
                const uint32_t off = (uint32_t)(min(r, nrows - 1) * D + c * 8) * 2u;
                lds_copy16(kp, off, (lds_ptr_t)(stage + (wave * KPW + u) * 1024));
            }
        }
    };
    // ... and its transposed values into stage `buf`'s V region.
    auto issue_exact_v = [&](int j, int buf) SOL_INLINE {
        j = __builtin_amdgcn_readfirstlane(j);
        char* stage = smem + buf * L::STAGE;
        const char* vp = reinterpret_cast<const char*>(a.vt + ((size_t)bh * a.NK + j) * D * kBlockK);
#pragma unroll
        for (int u = 0; u < VPW; ++u)
            lds_copy16(vp, vofs(u), (lds_ptr_t)(stage + L::KBYTES + (wave * VPW + u) * 1024));
    };

    const float cl = a.c_log2;

    // ---- building blocks of a tile -------------------------------------------------------
    // LDS operand addresses: per lane, the chunk read at k-step ks of a K tile and at k-step
    // kk of a V^T tile (rows r32 and 32+r32 of K share the swizzle; the second M-tile is a
    // constant 8 KB further, V^T M-tiles 4 KB apart).  With the stage fixed at compile time
    // every operand read is base register + immediate offset.  Under the key split a wave reads
    // K rows kbase.. and the V^T k-steps of its key half.
    constexpr int KT1 = 32 * L::KCPR * 16;   // byte offset of K rows 32..63
    uint32_t kadr[NKS], vadr[NPB];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kadr[ks] = 16u * (uint32_t)L::kpos(r32, 2 * ks + hh) + (uint32_t)(kh * KT1);
#pragma unroll
    for (int kk = 0; kk < NPB; ++kk)
        vadr[kk] = (uint32_t)L::KBYTES + 16u * (uint32_t)L::vpos(r32, 2 * (kk + NPB * kh) + hh);
    constexpr int VMT = 32 * L::VCPR * 16;   // byte offset between V^T M-tiles
    // Correction PV: the A operand (value means transposed: 32 values of d x 8 slots) of
    // M-tile mt and k-step kk comes from two transposed reads, slots 16kk + 4hh + 0..3 and
    // 16kk + 8 + 4hh + 0..3 (the slot order of the score registers); this lane reads row
    // 4hh + (lane%16)/4 (+16kk, +8) at d = 32mt + 16*((lane/16)%2) + 4*(lane%4).  The row
    // swizzle depends only on the row modulo 4, so kk and the second read add whole rows.
    uint32_t vtr[NDT];
    {
        const int s0 = 4 * hh + ((lane & 15) >> 2);
#pragma unroll
        for (int mt = 0; mt < NDT; ++mt) {
            const int cc = 4 * mt + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
            vtr[mt] = (uint32_t)(L::KBYTES + (s0 + kbase) * 2 * D + 16 * (cc ^ L::rswz(s0)) + 8 * (lane & 1));
        }
    }
    auto ldv_apx = [&](int kk, int mt, int soff) SOL_INLINE -> f16x8 {
        const char* p = smem + vtr[mt] + soff + kk * 16 * 2 * D;
        const s16x4 lo = lds_read_tr16(p);
        const s16x4 hi = lds_read_tr16(p + 8 * 2 * D);
        const s16x8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(f16x8, both);
    };

    // S^T = K Q^T over two 32-key M-tiles, operands double-buffered in registers.  Exact
    // tiles: bf16 keys x bf16 queries.  Correction tiles: f16 pooled keys x f16 queries, so the
    // pooled keys keep 11 significant bits.
    auto qk = [&](auto apx_tag, auto stage_tag, const auto& qop, f32x16& s0, f32x16& s1) SOL_INLINE {
        constexpr bool APX = decltype(apx_tag)::value;
        constexpr int SOFF = decltype(stage_tag)::value * L::STAGE;
        using AT = std::conditional_t<APX, f16x8, bf16x8>;
        AT a0[2], a1[2];
        a0[0] = *reinterpret_cast<const AT*>(smem + kadr[0] + SOFF);
        if constexpr (NS == 2) a1[0] = *reinterpret_cast<const AT*>(smem + kadr[0] + SOFF + KT1);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            if (ks + 1 < NKS) {
                a0[(ks + 1) & 1] = *reinterpret_cast<const AT*>(smem + kadr[ks + 1] + SOFF);
                if constexpr (NS == 2) a1[(ks + 1) & 1] = *reinterpret_cast<const AT*>(smem + kadr[ks + 1] + SOFF + KT1);
            }
            if constexpr (APX) {
                s0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a0[ks & 1], qop[ks], s0, 0, 0, 0);
                if constexpr (NS == 2) s1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a1[ks & 1], qop[ks], s1, 0, 0, 0);
            } else {
                s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[ks & 1], qop[ks], s0, 0, 0, 0);
                if constexpr (NS == 2) s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[ks & 1], qop[ks], s1, 0, 0, 0);
            }
        }
    };
    // Keys past the end of the sequence (only in the last key block) -> -inf.
    auto mask_tail = [&](int j, f32x16& s0, f32x16& s1) SOL_INLINE {
        const int nvalid = a.N - j * kBlockK - kbase;
        if (nvalid < kBlockK - kbase) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int key0 = 8 * (r >> 2) + 4 * hh + (r & 3);
                if (key0 >= nvalid) s0[r] = kNegInf;
                if (NS == 2 && 32 + key0 >= nvalid) s1[r] = kNegInf;
            }
        }
    };
    // Causal mask of a partially visible key block j: keys at or past this lane's limit -> -inf.
    auto mask_causal = [&](int j, f32x16& s0, f32x16& s1) SOL_INLINE {
        const int rel = qlim - j * kBlockK - kbase;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int key0 = 8 * (r >> 2) + 4 * hh + (r & 3);
            if (key0 >= rel) s0[r] = kNegInf;
            if (NS == 2 && 32 + key0 >= rel) s1[r] = kNegInf;
        }
    };
    // Correction tile of chunk c: slot j contributes with log2(n_j) (the multiplicity of Eq.
    // solattn_denominator) unless it is selected (exact tile) or past the routable keys.
    auto bias_apx = [&](int c, f32x16& s0, f32x16& s1) SOL_INLINE {
        // Element r of this lane's score registers holds slot 4*hh + off(r) (s0) or 32 + that
        // (s1), off(r) = 8*(r/4) + r%4.  Slots below nv are unselected routable blocks and take
        // the multiplicity bias (log2 n_j); the rest of the last tile is padding.
        int nv = nuns - c * kChunk - 4 * hh - kbase;      // off() bound of the valid slots
        int last = last_slot - c * kChunk - 4 * hh - kbase;
        // opaque here, so that the 32 biases are formed where they are added and not hoisted
        // into the MFMA slots of the iteration, where they would hold 32 registers
        asm volatile("" : "+v"(nv), "+v"(last));
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int off = 8 * (r >> 2) + (r & 3);
            const float b0 = (off == last) ? a.bias_last : a.bias_full;
            const float b1 = (off + 32 == last) ? a.bias_last : a.bias_full;
            s0[r] += off < nv ? b0 : kNegInf;
            if constexpr (NS == 2) s1[r] += off + 32 < nv ? b1 : kNegInf;
        }
    };
    // Online softmax in the log2 domain with lazy rescaling, split so that the (rarely
    // taken) rescale branch sits apart from the MFMA/VALU stream:
    //   tile_max  - row max of a score tile (both lane halves of a query agree)
    //   rescale   - raise the running max (log2 units) if a tile's max exceeds it by more than
    //               kRescaleSlack
    //   exps      - P^T = exp2(S*c + bo - m) packed as f16 B operands; row sums from the rounded
    //               P.  bo is a per-tile exponent offset: log2(64) for correction tiles whose
    //               64 slots are all full routable blocks (their multiplicity), else 0.
    auto tile_max = [&](const f32x16& s0, const f32x16& s1) SOL_INLINE -> float {
        // balanced tree of three-input maxima over the lane's 32 (16 under the key split)
        // scores (v_max3: 17 instructions for 32, short dependency chains) ...
        float m0;
        if constexpr (NS == 2) {
            float x[32];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                x[r] = s0[r];
                x[16 + r] = s1[r];
            }
            float a3[11];
#pragma unroll
            for (int i = 0; i < 10; ++i) a3[i] = fmaxf(fmaxf(x[3 * i], x[3 * i + 1]), x[3 * i + 2]);
            a3[10] = fmaxf(x[30], x[31]);
            const float b0 = fmaxf(fmaxf(a3[0], a3[1]), a3[2]), b1 = fmaxf(fmaxf(a3[3], a3[4]), a3[5]);
            const float b2 = fmaxf(fmaxf(a3[6], a3[7]), a3[8]), b3 = fmaxf(a3[9], a3[10]);
            m0 = fmaxf(fmaxf(fmaxf(b0, b1), b2), b3);
        } else {
            float a3[5];
#pragma unroll
            for (int i = 0; i < 5; ++i) a3[i] = fmaxf(fmaxf(s0[3 * i], s0[3 * i + 1]), s0[3 * i + 2]);
            const float b0 = fmaxf(fmaxf(a3[0], a3[1]), a3[2]), b1 = fmaxf(fmaxf(a3[3], a3[4]), s0[15]);
            m0 = fmaxf(b0, b1);
        }
        // ... then across the lane pair (l, l+32) that holds the query's other 32 keys, with a
        // VALU lane swap instead of an LDS permute
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(m0), __float_as_uint(m0), false, false);
        return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    };
    auto rescale = [&](float mt_) SOL_INLINE {
        const bool need = mt_ > m_run + kRescaleSlack;
        if (__ballot(need)) {
            const float mnew = need ? mt_ : m_run;
            const float alpha = (m_run == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(m_run - mnew);
#pragma unroll
            for (int mt = 0; mt < NDT; ++mt) o[mt] *= alpha;
#pragma unroll
            for (int u = 0; u < 4; ++u) l_run[u] *= alpha;
            m_run = mnew;
        }
    };
    auto exps = [&](const f32x16& s0, const f32x16& s1, f16x8 (&pb)[NPB], float bo) SOL_INLINE {
        const float msub = (m_run == kNegInf ? 0.f : m_run) - bo;
        const f16x2 ones = {(_Float16)1.f, (_Float16)1.f};
#pragma unroll
        for (int tt = 0; tt < NS; ++tt) {
#pragma unroll
            for (int sh = 0; sh < 2; ++sh) {
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const int r = 8 * sh + e;
                    const float x0 = tt ? s1[r] : s0[r];
                    const float x1 = tt ? s1[r + 1] : s0[r + 1];
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(x0, cl, -msub));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(x1, cl, -msub));
                    const f16x2 pp = {(_Float16)p0, (_Float16)p1};
                    l_run[2 * tt + sh] = __builtin_amdgcn_fdot2(pp, ones, l_run[2 * tt + sh], false);
                    pb[2 * tt + sh][e] = pp[0];
                    pb[2 * tt + sh][e + 1] = pp[1];
                }
            }
        }
    };
    auto softmax = [&](const f32x16& s0, const f32x16& s1, f16x8 (&pb)[NPB], float bo) SOL_INLINE {
        rescale(tile_max(s0, s1) * cl + bo);
        exps(s0, s1, pb, bo);
    };
    // O^T += V^T P^T, operands double-buffered in registers.
    auto pv = [&](auto apx_tag, auto stage_tag, const f16x8 (&pb)[NPB]) SOL_INLINE {
        constexpr bool APX = decltype(apx_tag)::value;
        constexpr int SOFF = decltype(stage_tag)::value * L::STAGE;
        auto ld = [&](int kk, int mt) SOL_INLINE -> f16x8 {
            if constexpr (APX) return ldv_apx(kk, mt, SOFF);
            else return *reinterpret_cast<const f16x8*>(smem + vadr[kk] + SOFF + mt * VMT);
        };
        f16x8 av[2];
        av[0] = ld(0, 0);
        // kk-major: consecutive MFMAs update different accumulators (no dependent issue)
#pragma unroll
        for (int i = 0; i < NDT * NPB; ++i) {
            const int kk = i / NDT, mt = i % NDT;
            if (i + 1 < NDT * NPB) av[(i + 1) & 1] = ld((i + 1) / NDT, (i + 1) % NDT);
            o[mt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av[i & 1], pb[kk], o[mt], 0, 0, 0);
        }
    };
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using APX_T = std::integral_constant<bool, true>;
    using EXACT_T = std::integral_constant<bool, false>;

    // ---- tile pipeline -------------------------------------------------------------------
    // Both kinds of tile run the same software pipeline, keys one tile ahead of values:
    // iteration t computes the scores of tile t+1 (MFMA) while the softmax of tile t (VALU)
    // runs, then O += V_t P_t.  Stage b's K region holds tile t+1 while its V region still
    // holds tile t, so both stages are busy without a third buffer.  The loop is unrolled by
    // two so that the stage of every LDS access is a compile-time offset.
    //   correction tiles (sparse mode, napx of them): 64 gathered unselected routable blocks,
    //     f16 pooled keys against the f16 query copy plus the multiplicity bias of each slot;
    //   exact tiles (ntiles of them): a bf16 key block against the bf16 queries.
    // The ragged last key block can only be the final exact tile (it is the last selected or
    // the last forced block), so its mask is applied after the loop.
    auto pipeline = [&](auto apx_tag, const auto& qop, const int T, auto code) SOL_INLINE {
        constexpr bool APX = decltype(apx_tag)::value;
        using KT = std::conditional_t<APX, f16x8, bf16x8>;
        // copies of the tile with code c (its key block, or its correction chunk)
        auto issue_k = [&](int c, int buf) SOL_INLINE {
            if constexpr (APX) issue_apx_k(c, buf);
            else issue_exact_k(c, buf);
        };
        auto issue_v = [&](int c, int buf) SOL_INLINE {
            if constexpr (APX) issue_apx_v(c, buf);
            else issue_exact_v(c, buf);
        };
        auto mfma_qk = [](const KT& av, const KT& bq, const f32x16& acc) SOL_INLINE {
            if constexpr (APX) return __builtin_amdgcn_mfma_f32_32x32x16_f16(av, bq, acc, 0, 0, 0);
            else return __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bq, acc, 0, 0, 0);
        };
        // scores of tile t are complete: returns the tile's exponent offset bo.  Correction
        // tiles: every tile but the last holds 64 unselected full blocks (the ragged last key
        // block, the largest index, and the padding slots can only be in the last tile), so
        // their multiplicity is the offset log2(64) and their scores stay untouched; the last
        // tile gets the per-slot bias after the loop.  Exact tiles: mask the keys a row does not
        // see (partially visible blocks under a causal mask).
        auto scores_done = [&](int t, int j, f32x16& s0, f32x16& s1) SOL_INLINE -> float {
            if constexpr (APX) {
                return t < T - 1 ? kLog2BlockK : 0.f;
            } else if constexpr (CAUSAL) {
                if (j >= nr) mask_causal(j, s0, s1);
            }
            return 0.f;
        };
        // row max of a finished score tile in log2 units, offset included
        auto tile_max_l2 = [&](const f32x16& s0, const f32x16& s1, float bo) SOL_INLINE -> float {
            const float m = tile_max(s0, s1) * cl;
            if constexpr (APX) return m + bo;
            else return m;
        };
        // Tile codes are read one step before their copies are issued, so that no list read
        // sits between a barrier and the copies and operand reads after it: entering step t,
        // cv = code(t+1) (its V goes out in step t) and ck = code(t+2) (its K goes out in step t).
        const int c0 = code(0);
        issue_k(c0, 0);
        issue_v(c0, 0);
        int cv = 0, ck = 0;
        if (T > 1) {
            cv = code(1);
            issue_k(cv, 1);
        }
        if (T > 2) ck = code(2);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        f32x16 s0 = f32x16{}, s1 = f32x16{};
        qk(apx_tag, S0{}, qop, s0, s1);
        float bo = scores_done(0, c0, s0, s1);   // offset of the tile whose scores are in s0/s1
        float mx = tile_max_l2(s0, s1, bo);
        // The first step refills stage 0's K region (tile 2) that QK^T(0) has just read; every
        // later refill of a region follows the barrier that ends the iteration which read it.
        if (T > 2) __syncthreads();
        // iteration t with t & 1 == P: K of tile t+1 in stage P^1, V of tile t in stage P
        // D = 128: one pipelined iteration as 32 MFMA slots.  Slots 0-15 run QK^T of tile t+1
        // while the exponentials of tile t are formed (one pair per slot, P block k in slots
        // 4k..4k+3); slots 16-31 run PV of tile t, which leaves their 16 MFMAs to hide the row
        // max of tile t+1 (finishing QK^T(t+1) early measured 1-2% faster than interleaving it
        // with PV(t)).  Successive MFMAs on one accumulator are at least two slots apart, and
        // operands are read from LDS two slots ahead.  Under the key split the same schedule has
        // 8 + 8 slots (one 32-key score tile, two P blocks).
        // Generic iteration (any D): the same work in source order.
        auto step_generic = [&](auto par_tag, int t) SOL_INLINE {
            constexpr int P = decltype(par_tag)::value;
            rescale(mx);
            if (t + 2 < T) issue_k(ck, P);
            issue_v(cv, P ^ 1);
            const int cn = t + 3 < T ? code(t + 3) : 0;
            f32x16 n0 = f32x16{}, n1 = f32x16{};
            qk(apx_tag, std::integral_constant<int, P ^ 1>{}, qop, n0, n1);
            f16x8 pb[NPB];
            exps(s0, s1, pb, bo);
            pv(apx_tag, par_tag, pb);
            bo = scores_done(t + 1, cv, n0, n1);
            mx = tile_max_l2(n0, n1, bo);
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            s0 = n0;
            s1 = n1;
            cv = ck;
            ck = cn;
        };
        auto step_slots = [&](auto par_tag, int t) SOL_INLINE {
            constexpr int P = decltype(par_tag)::value;
            constexpr int KOFF = (P ^ 1) * L::STAGE;   // K of tile t+1
            constexpr int VOFF = P * L::STAGE;         // V of tile t
            rescale(mx);
            if (t + 2 < T) issue_k(ck, P);
            issue_v(cv, P ^ 1);
            const int cn = t + 3 < T ? code(t + 3) : 0;
            const float msub = (m_run == kNegInf ? 0.f : m_run) - bo;
            const f16x2 ones = {(_Float16)1.f, (_Float16)1.f};
            // Row sums of the rounded P.  Non-causal kernels: the f16 dot product, right after the
            // pair's exponentials (beside the QK^T MFMAs; in the PV slots it stalls the matrix
            // pipe, 3-5% slower).  Causal kernels: two mixed FMAs per pair in the PV slots, 4%
            // faster there than the dot product (their register use and schedule differ).
            constexpr bool kRowSumInPV = CAUSAL;
            f16x8 pb[NPB];
            auto exp_pair = [&](int kk, int q) SOL_INLINE {   // elements 2q, 2q+1 of P block kk
                const int tt = kk >> 1, r = 8 * (kk & 1) + 2 * q;
                const float x0 = tt ? s1[r] : s0[r];
                const float x1 = tt ? s1[r + 1] : s0[r + 1];
                const float p0 = __builtin_amdgcn_exp2f(fmaf(x0, cl, -msub));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(x1, cl, -msub));
                const f16x2 pp = {(_Float16)p0, (_Float16)p1};
                if constexpr (!kRowSumInPV) l_run[kk] = __builtin_amdgcn_fdot2(pp, ones, l_run[kk], false);
                pb[kk][2 * q] = pp[0];
                pb[kk][2 * q + 1] = pp[1];
            };
            // slot -> operation: slots 0..NQK-1 QK^T (index i: k-step i/NS, key half i%NS), the
            // rest PV (index i: k-step i/4, d M-tile i%4).  Under the key split a wave has 8 + 8
            // slots, each of the first 8 with one exponential pair.
            constexpr int NQK = NKS * NS, NSLOT = NQK + NPB * NDT;
            auto kind = [](int sl) SOL_INLINE { return sl < NQK ? 0 : 1; };
            auto index = [](int sl) SOL_INLINE { return sl < NQK ? sl : sl - NQK; };
            auto ldk = [&](int qi) SOL_INLINE {
                if constexpr (NS == 1) return *reinterpret_cast<const KT*>(smem + kadr[qi] + KOFF);
                else return *reinterpret_cast<const KT*>(smem + kadr[qi >> 1] + KOFF + (qi & 1) * KT1);
            };
            auto ldv = [&](int pi) SOL_INLINE -> f16x8 {
                if constexpr (APX) return ldv_apx(pi >> 2, pi & 3, VOFF);
                else return *reinterpret_cast<const f16x8*>(smem + vadr[pi >> 2] + VOFF + (pi & 3) * VMT);
            };
            KT kop[4];
            f16x8 vop[4];
            int nk = 0, nv = 0;   // operands loaded so far (ring of 4)
            auto prefetch = [&](int sl) SOL_INLINE {
                if (sl >= NSLOT) return;
                if (kind(sl) == 0) kop[(nk++) & 3] = ldk(index(sl));
                else vop[(nv++) & 3] = ldv(index(sl));
            };
            f32x16 n0 = f32x16{}, n1 = f32x16{};
            prefetch(0);
            prefetch(1);
            int uk = 0, uv = 0;   // operands consumed so far
#pragma unroll
            for (int sl = 0; sl < NSLOT; ++sl) {
                // Wave priority: highest in the QK^T half (the exponentials), lower in the PV half,
                // lowest outside the tile loops (routing, epilogue), which the other workgroup on the
                // CU can then overlap: 1-2.4% faster in the sparse modes, dense within noise.  Under
                // the key split (8 + 8 slots) the PV half goes first instead: 1.5% faster there.
                constexpr int kPrioQK = NS == 1 ? 1 : 2, kPrioPV = NS == 1 ? 2 : 1;
                if (sl == 0) __builtin_amdgcn_s_setprio(kPrioQK);
                if (sl == NQK) __builtin_amdgcn_s_setprio(kPrioPV);
                prefetch(sl + 2);
                const int id = index(sl);
                if (kind(sl) == 0) {
                    const KT av = kop[(uk++) & 3];
                    if (NS == 1) n0 = mfma_qk(av, qop[id], n0);
                    else if (id & 1) n1 = mfma_qk(av, qop[id >> 1], n1);
                    else n0 = mfma_qk(av, qop[id >> 1], n0);
                } else {
                    const f16x8 av = vop[(uv++) & 3];
                    o[id & 3] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, pb[id >> 2], o[id & 3], 0, 0, 0);
                }
                if (sl < 4 * NPB) exp_pair(sl >> 2, sl & 3);
                // row max of tile t+1 in the second-last slot (0.2-0.8% faster than after the last;
                // the causal kernels take it after the loop: their masked form inside the
                // unrolled loop multiplies the code)
                if constexpr (!CAUSAL) {
                    if (sl == NSLOT - 2) {
                        bo = scores_done(t + 1, cv, n0, n1);
                        mx = tile_max_l2(n0, n1, bo);
                    }
                }
                if constexpr (kRowSumInPV) {
                    if (sl >= NQK && sl - NQK < 4 * NPB) {   // pair sl - NQK, while its P block is read
                        const int kk = (sl - NQK) >> 2, q = (sl - NQK) & 3;
                        l_run[kk] = add_f16x2(l_run[kk], f16x2{pb[kk][2 * q], pb[kk][2 * q + 1]});
                    }
                }
                // Each slot is its own scheduling region: left free, the scheduler sinks the
                // exponentials towards their PV consumers and leaves most QK^T MFMAs of the
                // wave with no VALU work beside them (1-2% slower, measured).
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (CAUSAL) {
                bo = scores_done(t + 1, cv, n0, n1);
                mx = tile_max_l2(n0, n1, bo);
            }
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            s0 = n0;
            s1 = n1;
            cv = ck;
            ck = cn;
        };
        auto step = [&](auto par_tag, int t) SOL_INLINE {
            if constexpr (D == 128) step_slots(par_tag, t);
            else step_generic(par_tag, t);
        };
        int t = 0;
        for (; t + 2 < T; t += 2) {
            step(S0{}, t);
            step(S1{}, t + 1);
        }
        if (t + 1 < T) {
            step(S0{}, t);
            ++t;
        }
        // last tile (t == T-1): its max is taken again here, after the bias or the tail mask
        if constexpr (APX) bias_apx(code(T - 1), s0, s1);
        else mask_tail(code(T - 1), s0, s1);
        f16x8 pb[NPB];
        softmax(s0, s1, pb, bo);
        if ((T - 1) & 1) pv(apx_tag, S1{}, pb);
        else pv(apx_tag, S0{}, pb);
    };

    if (MODE == kSparse && napx > 0) {
        f16x8 qh[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const bf16x8 qv = qrow < a.N ? *reinterpret_cast<const bf16x8*>(qrow_p + 16 * ks) : bf16x8{};
#pragma unroll
            for (int e = 0; e < 8; ++e) qh[ks][e] = (_Float16)(float)qv[e];
        }
        __builtin_amdgcn_s_setprio(1);
        pipeline(APX_T{}, qh, napx, [&](int t) SOL_INLINE { return t; });
        __builtin_amdgcn_s_setprio(0);
        __syncthreads();   // the stages are refilled below while the last V tile may still be read
    }
    const int T = ntiles;
    if (T > 0) {
        bf16x8 qf[NKS];
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
            qf[ks] = qrow < a.N ? *reinterpret_cast<const bf16x8*>(qrow_p + 16 * ks) : bf16x8{};
        __builtin_amdgcn_s_setprio(1);
        pipeline(EXACT_T{}, qf, T, [&](int t) SOL_INLINE { return tile_code(t); });
        __builtin_amdgcn_s_setprio(0);
    }

    // ---- epilogue: O = O^T / l, bf16
    const float lsum = (l_run[0] + l_run[1]) + (l_run[2] + l_run[3]);
    const float lt = lsum + __shfl_xor(lsum, 32);
    uint16_t* op = a.out + ((size_t)bh * a.N + qrow) * D;   // written only for rows < N
    auto store = [&](int mt, const f32x16& v, float inv) SOL_INLINE {   // d rows 32mt.. of O^T
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int d0 = 32 * mt + 8 * i + 4 * hh;
            uint32_t w0 = (uint32_t)f32_to_bf16_bits(v[4 * i + 0] * inv) |
                          ((uint32_t)f32_to_bf16_bits(v[4 * i + 1] * inv) << 16);
            uint32_t w1 = (uint32_t)f32_to_bf16_bits(v[4 * i + 2] * inv) |
                          ((uint32_t)f32_to_bf16_bits(v[4 * i + 3] * inv) << 16);
            *reinterpret_cast<uint2*>(op + d0) = make_uint2(w0, w1);
        }
    };
    if constexpr (!KSPLIT) {
        const float inv = lt > 0.f ? 1.0f / lt : 0.f;
        if (qrow < a.N) {
#pragma unroll
            for (int mt = 0; mt < NDT; ++mt) store(mt, o[mt], inv);
        }
    } else {
        // The two key halves of a row hold separate softmax states (m, l, O) over disjoint keys.
        // Wave (rw, kh) finishes d M-tiles 2kh and 2kh+1: it hands its other two M-tiles, its
        // running max and its row sum to its partner (rw, 1-kh) through LDS (the tile stages are
        // free once every wave is past its last PV), takes the partner's copy of its own two, and
        // rescales both states to the common max: O = (a0 O0 + a1 O1) / (a0 l0 + a1 l1).
        static_assert(NDT == 4, "the key split assumes d = 128");
        constexpr int XREG = 2 * 16 * 64 + 2 * 64;   // floats per wave: 2 M-tiles, m, l
        static_assert(4 * XREG * 4 <= 2 * L::STAGE, "exchange buffer exceeds the tile stages");
        float* xbuf = reinterpret_cast<float*>(smem);
        __syncthreads();
        float* mine = xbuf + wave * XREG;
        auto put = [&](const f32x16& v0, const f32x16& v1) SOL_INLINE {   // lane-contiguous 16 B
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                *reinterpret_cast<float4*>(mine + (i * 64 + lane) * 4) = make_float4(v0[4 * i], v0[4 * i + 1], v0[4 * i + 2], v0[4 * i + 3]);
                *reinterpret_cast<float4*>(mine + ((4 + i) * 64 + lane) * 4) = make_float4(v1[4 * i], v1[4 * i + 1], v1[4 * i + 2], v1[4 * i + 3]);
            }
        };
        if (kh == 0) put(o[2], o[3]);
        else put(o[0], o[1]);
        mine[2048 + lane] = m_run;
        mine[2048 + 64 + lane] = lt;
        __syncthreads();
        const float* theirs = xbuf + (wave ^ 2) * XREG;
        const float mp = theirs[2048 + lane], lp = theirs[2048 + 64 + lane];
        const float mm = fmaxf(m_run, mp);
        const float a0 = m_run == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m_run - mm);
        const float a1 = mp == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mp - mm);
        const float l = a0 * lt + a1 * lp;
        const float inv = l > 0.f ? 1.0f / l : 0.f;
        auto merged = [&](const f32x16& own, int half) SOL_INLINE -> f32x16 {
            f32x16 r;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 p = *reinterpret_cast<const float4*>(theirs + ((4 * half + i) * 64 + lane) * 4);
                r[4 * i + 0] = a0 * own[4 * i + 0] + a1 * p.x;
                r[4 * i + 1] = a0 * own[4 * i + 1] + a1 * p.y;
                r[4 * i + 2] = a0 * own[4 * i + 2] + a1 * p.z;
                r[4 * i + 3] = a0 * own[4 * i + 3] + a1 * p.w;
            }
            return r;
        };
        if (qrow < a.N) {
            if (kh == 0) {
                store(0, merged(o[0], 0), inv);
                store(1, merged(o[1], 1), inv);
            } else {
                store(2, merged(o[2], 0), inv);
                store(3, merged(o[3], 1), inv);
            }
        }
    }
}

// The fused kernel runs persistent workgroups (as many as fit on the device at once) that
// claim query blocks from eight queues, one per XCD.  Queue x lists, in order, the blocks of
// a fixed XCD-aware assignment: 2^hlog heads at a time, each on 8 >> hlog XCDs, and queue x
// holds a contiguous range of per_x blocks of its head (through the query-block order in the
// sparse modes), so the workgroups resident on one XCD work through neighbouring blocks of one
// head and share its K/V in their L2.  Under a causal mask the work of a query block grows with its index, so the
// head's blocks are cut into 16 segments and queue x takes segment 15 - x (descending, the
// longer blocks first) and then segment x.  Consecutive workgroups go round-robin to the 8
// XCDs, so workgroup w serves queue w & 7 first; once that queue is empty it takes blocks
// from the queue with the most left.  XCDs whose blocks need more tiles, or that run slower,
// thus get help at the end instead of finishing last.  A block's result does not depend on
// which workgroup computes it, and every claim either takes a block or finds a queue empty
// for good, so each workgroup stops after at most eight failed claims.
template <int D, int BQ, int MODE, bool CAUSAL>
__global__ __launch_bounds__((kAttnThreads<D, BQ>)) __attribute__((amdgpu_waves_per_eu(2, 2)))
void routed_attn_kernel(AttnArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ int s_task[2];
    const int home = blockIdx.x & 7;
    const unsigned groups = CAUSAL ? (unsigned)a.BH : (unsigned)((a.BH + (1 << a.hlog) - 1) >> a.hlog);
    const unsigned qlen = (unsigned)a.per_x * groups;   // positions per queue
    for (;;) {
        __syncthreads();   // the previous block is done with LDS and with s_task
        // Claims are made when a block starts, not ahead of it: a queue position then also
        // orders the blocks by start time, which the exact tiles' start phase relies on.
        if (threadIdx.x == 0) {
            int tx = -1;
            unsigned tp = 0;
            const unsigned p = atomicAdd(a.queue + 32 * home, 1u);
            if (p < qlen) {
                tx = home;
                tp = p;
            } else {
                for (int tries = 0; tries < 8 && tx < 0; ++tries) {
                    int best = -1;
                    unsigned left = 0;
                    for (int x = 0; x < 8; ++x) {
                        const unsigned c = __hip_atomic_load(a.queue + 32 * x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if (c < qlen && qlen - c > left) {
                            left = qlen - c;
                            best = x;
                        }
                    }
                    if (best < 0) break;
                    const unsigned q = atomicAdd(a.queue + 32 * best, 1u);
                    if (q < qlen) {
                        tx = best;
                        tp = q;
                    }
                }
            }
            s_task[0] = tx;
            s_task[1] = (int)tp;
        }
        __syncthreads();
        const int x = s_task[0], y = s_task[1];
        if (x < 0) return;
        int bh, qi;
        if constexpr (CAUSAL) {
            bh = y / a.per_x;
            const int u = y % a.per_x, hp = a.per_x >> 1;
            qi = u < hp ? (15 - x) * hp + (hp - 1 - u) : x * hp + (u - hp);
        } else {
            // 2^hlog heads at a time, each on 8 >> hlog XCDs: queue x serves head (x >> gl) of
            // the current group, blocks (x mod 2^gl)*per_x ..
            const int gl = 3 - a.hlog;
            bh = ((y / a.per_x) << a.hlog) + (x >> gl);
            qi = (x & ((1 << gl) - 1)) * a.per_x + (y % a.per_x);
            if (a.order != nullptr && bh < a.BH && qi < a.NQ) qi = a.order[(size_t)bh * a.NQ + qi];
        }
        if (bh < a.BH && qi < a.NQ) attn_block<D, BQ, MODE, CAUSAL>(a, smem, bh, qi, y);
    }
}

__global__ void queue_reset_kernel(uint32_t* q) {
    if (threadIdx.x < 8) q[32 * threadIdx.x] = 0u;
}

// ---------------------------------------------------------------------------
// Routed attention with f32 inputs (correctness-first path, VALU only).  One thread per
// query row; K/V (or pooled Kbar/Vbar for correction tiles) staged in LDS one tile at a
// time; per-key streaming softmax in natural-exp units.
// ---------------------------------------------------------------------------
struct AttnArgsF32 {
    const float* q;
    const float* k;
    const float* v;
    const float* qbar;
    const float* kbar;
    const float* vbar;
    const float* tau;
    float* out;
    uint32_t* blkcount;
    uint32_t* mask_out;
    int BH, N, NQ, NK, NKr, NC, MW;
    float scale;
    int causal_g;
    float beta;
};

template <int D, int BQ, int MODE, bool CAUSAL>
__global__ __launch_bounds__(BQ) void routed_attn_f32_kernel(AttnArgsF32 a) {
    constexpr int NT = BQ;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    float* ks = reinterpret_cast<float*>(smem);            // [64][D]
    float* vs = ks + kBlockK * D;                          // [64][D]
    float* qt = vs + kBlockK * D;                          // [D][BQ]
    char* rest = reinterpret_cast<char*>(qt + D * BQ);
    int* scan_scratch = reinterpret_cast<int*>(rest);
    uint32_t* selw = reinterpret_cast<uint32_t*>(rest + 64);
    uint16_t* list = reinterpret_cast<uint16_t*>(rest + 64 + 4 * ((a.MW + 3) & ~3));
    int* wpre = reinterpret_cast<int*>(rest + ((64 + 4 * ((a.MW + 3) & ~3) + 2 * (a.NC * kChunk + a.NK) + 15) & ~15));
    float* prox = reinterpret_cast<float*>(wpre + ((a.MW + 3) & ~3));   // after the word prefixes
    const uint16_t* ulist = list;            // correction slots (unselected routable blocks, padded)
    const uint16_t* elist = list + a.NC * kChunk;   // exact tiles

    const int bh = blockIdx.y, qi = blockIdx.x, tid = threadIdx.x;
    int nr = a.NKr, ne = a.NK;               // routable blocks [0, nr), forced blocks [nr, ne)
    if constexpr (CAUSAL) causal_ranges<BQ>(qi, a.causal_g, a.N, a.NK, nr, ne);
    int ntiles, nsel, nuns = 0;
    if (MODE == kDense) {
        ntiles = ne;
        nsel = nr;
    } else {
        const float tau_i = CAUSAL ? 0.f : a.tau[(size_t)bh * a.NQ + qi];
        ntiles = route_and_list<D, NT, MODE, CAUSAL>(a.qbar + ((size_t)bh * a.NQ + qi) * D,
                                                     a.kbar + (size_t)bh * a.NK * D, tau_i, a.beta, a.scale, a.NKr,
                                                     nr, ne, a.MW, prox, selw, list, a.NC * kChunk, scan_scratch,
                                                     wpre, &nuns, &nsel);
        if (a.mask_out)
            for (int w = tid; w < a.MW; w += NT) a.mask_out[((size_t)bh * a.NQ + qi) * a.MW + w] = selw[w];
    }
    if (tid == 0) a.blkcount[(size_t)bh * a.NQ + qi] = (uint32_t)nsel;

    const int row = qi * BQ + tid;
    const int qlim = CAUSAL ? causal_lim(row, a.causal_g, a.N) : a.N;   // this row sees keys < qlim
    for (int e = tid; e < BQ * D; e += NT) {
        const int rr = e / D, c = e % D, gr = qi * BQ + rr;
        qt[c * BQ + rr] = gr < a.N ? a.q[((size_t)bh * a.N + gr) * D + c] : 0.f;
    }
    float o[D];
#pragma unroll
    for (int c = 0; c < D; ++c) o[c] = 0.f;
    float m = kNegInf, l = 0.f;

    // correction tiles first (64 unselected routable blocks each), then the exact tiles
    const int napx = MODE == kSparse ? (nuns + kChunk - 1) / kChunk : 0;
    for (int n = 0; n < napx + ntiles; ++n) {
        const bool apx = n < napx;
        const int c = apx ? n : (MODE == kDense ? n : (int)elist[n - napx]);
        __syncthreads();
        for (int e = tid; e < kBlockK * D; e += NT) {
            const int rr = e / D, cc = e % D;
            float kv = 0.f, vv = 0.f;
            if (apx) {
                const int u = c * kChunk + rr;
                if (u < nuns) {
                    const int j = ulist[u];
                    kv = a.kbar[((size_t)bh * a.NK + j) * D + cc];
                    vv = a.vbar[((size_t)bh * a.NK + j) * D + cc];
                }
            } else {
                const int gr = c * kBlockK + rr;
                if (gr < a.N) {
                    kv = a.k[((size_t)bh * a.N + gr) * D + cc];
                    vv = a.v[((size_t)bh * a.N + gr) * D + cc];
                }
            }
            ks[e] = kv;
            vs[e] = vv;
        }
        __syncthreads();
        for (int u = 0; u < kBlockK; ++u) {
            float bias = 0.f;
            if (apx) {
                if (c * kChunk + u >= nuns) continue;
                const int j = ulist[c * kChunk + u];
                bias = logf((float)min(kBlockK, a.N - j * kBlockK));
            } else if (c * kBlockK + u >= (CAUSAL && c >= nr ? qlim : a.N)) {
                continue;
            }
            float dot = 0.f;
#pragma unroll 16
            for (int cc = 0; cc < D; ++cc) dot = fmaf(qt[cc * BQ + tid], ks[u * D + cc], dot);
            const float s = dot * a.scale + bias;
            if (s > m) {
                const float alpha = m == kNegInf ? 0.f : expf(m - s);
                l *= alpha;
#pragma unroll
                for (int cc = 0; cc < D; ++cc) o[cc] *= alpha;
                m = s;
            }
            const float p = expf(s - m);
            l += p;
#pragma unroll
            for (int cc = 0; cc < D; ++cc) o[cc] = fmaf(p, vs[u * D + cc], o[cc]);
        }
    }
    if (row < a.N) {
        const float inv = l > 0.f ? 1.0f / l : 0.f;
        float* op = a.out + ((size_t)bh * a.N + row) * D;
#pragma unroll
        for (int cc = 0; cc < D; ++cc) op[cc] = o[cc] * inv;
    }
}

__global__ __launch_bounds__(256) void count_reduce_kernel(const uint32_t* __restrict__ blk, uint32_t* __restrict__ counts,
                                                           int NQ) {
    __shared__ uint32_t red[4];
    const int bh = blockIdx.x, t = threadIdx.x;
    uint32_t s = 0;
    for (int i = t; i < NQ; i += 256) s += blk[(size_t)bh * NQ + i];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
    if ((t & 63) == 0) red[t >> 6] = s;
    __syncthreads();
    if (t == 0) counts[bh] = red[0] + red[1] + red[2] + red[3];
}

template <typename K>
hipError_t allow_lds(K kernel, size_t bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

template <int D, int BQ, int MODE, bool CAUSAL>
hipError_t launch_attn_bf16(const Shape& s, const AttnArgs& a, hipStream_t st) {
    const size_t lds = attn_lds_bytes(s);
    auto kern = routed_attn_kernel<D, BQ, MODE, CAUSAL>;
    hipError_t e = allow_lds(kern, lds);
    if (e != hipSuccess) return e;
    // persistent grid: as many workgroups as fit at once, a multiple of 8 (one share per XCD),
    // never more than there are query-block positions
    int dev = 0, cus = 0, occ = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, kAttnThreads<D, BQ>, lds)) != hipSuccess) return e;
    const long long groups = CAUSAL ? a.BH : ((a.BH + (1 << a.hlog) - 1) >> a.hlog);
    const long long positions = 8LL * a.per_x * groups;
    long long grid = ((long long)std::max(cus * std::max(occ, 1), 8) / 8) * 8;
    grid = std::min(grid, positions);
    AttnArgs b = a;
    b.resident = (int)(grid / 8);
    kern<<<dim3((unsigned)grid), dim3(kAttnThreads<D, BQ>), lds, st>>>(b);
    return hipGetLastError();
}

template <int D, int BQ, int MODE, bool CAUSAL>
hipError_t launch_attn_f32(const Shape& s, const AttnArgsF32& a, hipStream_t st) {
    const size_t lds = attn_lds_bytes(s);
    auto kern = routed_attn_f32_kernel<D, BQ, MODE, CAUSAL>;
    hipError_t e = allow_lds(kern, lds);
    if (e != hipSuccess) return e;
    kern<<<dim3(a.NQ, a.BH), dim3(BQ), lds, st>>>(a);
    return hipGetLastError();
}

template <int D, int BQ, bool CAUSAL>
hipError_t dispatch_bf16_mode(const Shape& s, const AttnArgs& a, hipStream_t st) {
    switch (s.mode) {
        case kDense: return launch_attn_bf16<D, BQ, kDense, CAUSAL>(s, a, st);
        case kSparse: return launch_attn_bf16<D, BQ, kSparse, CAUSAL>(s, a, st);
        default: return launch_attn_bf16<D, BQ, kSparseNoCorr, CAUSAL>(s, a, st);
    }
}

template <int D, int BQ>
hipError_t dispatch_bf16(const Shape& s, const AttnArgs& a, hipStream_t st) {
    return s.causal ? dispatch_bf16_mode<D, BQ, true>(s, a, st) : dispatch_bf16_mode<D, BQ, false>(s, a, st);
}

template <int D, int BQ, bool CAUSAL>
hipError_t dispatch_f32_mode(const Shape& s, const AttnArgsF32& a, hipStream_t st) {
    switch (s.mode) {
        case kDense: return launch_attn_f32<D, BQ, kDense, CAUSAL>(s, a, st);
        case kSparse: return launch_attn_f32<D, BQ, kSparse, CAUSAL>(s, a, st);
        default: return launch_attn_f32<D, BQ, kSparseNoCorr, CAUSAL>(s, a, st);
    }
}

template <int D, int BQ>
hipError_t dispatch_f32(const Shape& s, const AttnArgsF32& a, hipStream_t st) {
    return s.causal ? dispatch_f32_mode<D, BQ, true>(s, a, st) : dispatch_f32_mode<D, BQ, false>(s, a, st);
}

}  // namespace

// ---------------------------------------------------------------------------
// Host-side launch helpers
// ---------------------------------------------------------------------------
Shape make_shape(int B, int H, int N, int d, int bq, int bk, int mode, int dtype, int keep_tail_tokens,
                 int causal_granule) {
    Shape s{};
    s.causal = causal_granule;
    s.B = B; s.H = H; s.N = N; s.d = d; s.bq = bq; s.bk = bk;
    s.mode = mode & ~kThresholdDiagonal; s.dtype = dtype;
    s.diag = (mode & kThresholdDiagonal) ? 1 : 0;
    s.forced = bk > 0 ? keep_tail_tokens / bk : 0;
    s.BH = B * H;
    s.NQ = bq > 0 ? (N + bq - 1) / bq : 0;
    s.NK = bk > 0 ? (N + bk - 1) / bk : 0;
    s.NKr = s.NK - s.forced;
    s.NC = (s.NKr + kChunk - 1) / kChunk;
    s.Npad = s.NK * kBlockK;
    s.MW = (s.NKr + 31) / 32;
    return s;
}

size_t attn_lds_bytes(const Shape& s) {
    // scan scratch, selection words, lists, then (16-byte aligned) the words' prefix counts
    size_t rest = 64 + 4 * (size_t)((s.MW + 3) & ~3) + 2 * ((size_t)s.NC * kChunk + s.NK);
    rest = ((rest + 15) & ~(size_t)15) + 4 * (size_t)((s.MW + 3) & ~3);
    if (s.dtype == kBF16) {
        const size_t stage = (size_t)kBlockK * s.d * 2 * 2;
        // proxies of a causal row: in the tile stages when they fit (the kernel decides alike)
        if (s.causal && s.mode != kDense && 4 * (size_t)s.NKr > 2 * stage) rest += 4 * (size_t)s.NKr;
        return 2 * stage + rest;
    }
    if (s.causal && s.mode != kDense) rest += 4 * (size_t)s.NKr;   // proxies of a row
    return (size_t)2 * kBlockK * s.d * 4 + (size_t)s.d * s.bq * 4 + rest;
}

size_t workspace_layout(const Shape& s, char* base, Workspace* ws) {
    size_t off = 0;
    auto take = [&](size_t bytes) -> char* {
        char* p = base ? base + off : nullptr;
        off += (bytes + 255) & ~(size_t)255;
        return p;
    };
    const size_t BH = s.BH, d = s.d;
    const bool routing = s.mode != kDense;
    Workspace w;
    if (routing) {
        w.qbar = reinterpret_cast<float*>(take(BH * s.NQ * d * 4));
        w.kbar = reinterpret_cast<float*>(take(BH * s.NK * d * 4));
        w.muk = reinterpret_cast<float*>(take(BH * d * 4));
        w.cov = reinterpret_cast<float*>(take(BH * d * d * 4));
        w.tau = reinterpret_cast<float*>(take(BH * s.NQ * 4));
        w.sigma = reinterpret_cast<float*>(take(BH * s.NQ * 4));
        w.order = reinterpret_cast<uint16_t*>(take(BH * s.NQ * 2));
        w.mom = reinterpret_cast<double*>(take(moments_scratch_bytes(s.BH, s.NKr, s.d)));
    }
    if (s.dtype == kBF16) {
        w.vt = reinterpret_cast<_Float16*>(take(BH * d * (size_t)s.Npad * 2));
        if (routing) {
            w.kbarh = reinterpret_cast<_Float16*>(take(BH * (size_t)s.NC * kChunk * d * 2));
            w.vbarh = reinterpret_cast<_Float16*>(take(BH * (size_t)s.NC * kChunk * d * 2));
        }
    } else if (s.mode == kSparse) {
        w.vbar = reinterpret_cast<float*>(take(BH * s.NK * d * 4));
    }
    w.blkcount = reinterpret_cast<uint32_t*>(take(BH * s.NQ * 4));
    if (s.dtype == kBF16) w.queue = reinterpret_cast<uint32_t*>(take(8 * 32 * 4));
    if (ws) *ws = w;
    return off;
}

hipError_t launch_pool_mean(const void* x, float* mean, int dtype, int BH, int N, int d, int blk, hipStream_t st) {
    const int nb = (N + blk - 1) / blk;
    if (dtype == kBF16)
        pool_mean_kernel<uint16_t><<<dim3(nb, BH), dim3(256), 0, st>>>(static_cast<const uint16_t*>(x), mean, N, d, blk, nb);
    else
        pool_mean_kernel<float><<<dim3(nb, BH), dim3(256), 0, st>>>(static_cast<const float*>(x), mean, N, d, blk, nb);
    return hipGetLastError();
}

size_t moments_scratch_bytes(int BH, int NKr, int d) {
    return (size_t)BH * mom_splits(BH, NKr) * ((size_t)d * d + d) * sizeof(double);
}

hipError_t launch_moments_final(const float* kbar, float* muk, float* cov, double* scratch, int BH, int NK, int NKr,
                                int d, hipStream_t st) {
    if (d == 128)
        moments_final_kernel<128><<<dim3(128 * 128 / 256, BH), dim3(256), 0, st>>>(kbar, scratch, muk, cov, NK, NKr,
                                                                                    mom_splits(BH, NKr));
    else
        moments_final_kernel<64><<<dim3(64 * 64 / 256, BH), dim3(256), 0, st>>>(kbar, scratch, muk, cov, NK, NKr,
                                                                                  mom_splits(BH, NKr));
    return hipGetLastError();
}

hipError_t launch_moments(const float* kbar, float* muk, float* cov, double* scratch, int BH, int NK, int NKr, int d,
                          hipStream_t st) {
    const int ns = mom_splits(BH, NKr);
    if (d == 128) moments_partial_kernel<128><<<dim3(ns, BH), dim3(256), 0, st>>>(kbar, scratch, NK, NKr, ns);
    else moments_partial_kernel<64><<<dim3(ns, BH), dim3(256), 0, st>>>(kbar, scratch, NK, NKr, ns);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_moments_final(kbar, muk, cov, scratch, BH, NK, NKr, d, st);
}

hipError_t launch_tau(const float* qbar, const float* muk, const float* cov, float* tau, float* mu, float* sigma,
                      int BH, int NQ, int d, float beta, int diag, hipStream_t st) {
    const float scale = 1.0f / sqrtf((float)d);
    const dim3 grid((NQ + 15) / 16, BH);
    if (d == 128) {
        if (diag) tau_kernel<128, true><<<grid, dim3(256), 0, st>>>(qbar, muk, cov, tau, mu, sigma, NQ, beta, scale);
        else tau_kernel<128, false><<<grid, dim3(256), 0, st>>>(qbar, muk, cov, tau, mu, sigma, NQ, beta, scale);
    } else {
        if (diag) tau_kernel<64, true><<<grid, dim3(256), 0, st>>>(qbar, muk, cov, tau, mu, sigma, NQ, beta, scale);
        else tau_kernel<64, false><<<grid, dim3(256), 0, st>>>(qbar, muk, cov, tau, mu, sigma, NQ, beta, scale);
    }
    return hipGetLastError();
}

// Heads whose query blocks are in the attention kernel's queues at once (log2).  The workgroups
// resident on one XCD share its L2, so each XCD should work through one head at a time; with
// all 8 XCDs on one head each gets only NQ/8 blocks of it.  Fewer XCDs per head give each XCD
// longer runs of one head, as far as the heads in flight keep their K/V tiles (bf16 K and f16
// V^T, 4*Npad*d bytes per head) within kMallBudget of the shared MALL.  Heads differ in their
// kept fraction, so the XCDs of one head may finish early; the queues' stealing evens that out.
constexpr double kMallBudget = 96.0 * 1024 * 1024;
template <int D>
hipError_t launch_order_d(const float* qbar, const float* cov, const float* sigma, uint16_t* order, int BH, int NQ,
                          hipStream_t st) {
    const dim3 grid(BH), block(256);
    if (NQ <= 256) order_kernel<D, 1><<<grid, block, 0, st>>>(qbar, cov, sigma, order, NQ);
    else if (NQ <= 512) order_kernel<D, 2><<<grid, block, 0, st>>>(qbar, cov, sigma, order, NQ);
    else if (NQ <= 1024) order_kernel<D, 4><<<grid, block, 0, st>>>(qbar, cov, sigma, order, NQ);
    else if (NQ <= 2048) order_kernel<D, 8><<<grid, block, 0, st>>>(qbar, cov, sigma, order, NQ);
    else order_kernel<D, 16><<<grid, block, 0, st>>>(qbar, cov, sigma, order, NQ);
    return hipGetLastError();
}

hipError_t launch_order(const float* qbar, const float* cov, const float* sigma, uint16_t* order, int BH, int NQ, int d,
                        hipStream_t st) {
    return d == 128 ? launch_order_d<128>(qbar, cov, sigma, order, BH, NQ, st)
                    : launch_order_d<64>(qbar, cov, sigma, order, BH, NQ, st);
}

int heads_in_flight_log2(const Shape& s) {
    const double kv = 4.0 * (double)s.Npad * s.d;
    int hl = 0;
    while (hl < 3 && (double)(2 << hl) * kv <= kMallBudget && (2 << hl) <= s.BH) ++hl;
    return hl;
}

hipError_t launch_forward(const Shape& s, const void* q, const void* k, const void* v, void* out, float beta,
                          const Workspace& ws, uint32_t* counts, uint32_t* mask_out, hipStream_t st,
                          hipEvent_t ev_start, hipEvent_t ev_stop) {
    const bool routing = s.mode != kDense;
    const int d = s.d;
    hipError_t e;
    const float scale = 1.0f / sqrtf((float)d);
    if (s.dtype == kBF16) {
        const int nj = routing ? (s.NC * kChunk > s.NK ? s.NC * kChunk : s.NK) : s.NK;
        const uint16_t* kk = static_cast<const uint16_t*>(k);
        const uint16_t* vv = static_cast<const uint16_t*>(v);
        if (d == 128)
            prep_kv_kernel<128><<<dim3(nj, s.BH), dim3(256), 0, st>>>(kk, vv, ws.kbar, ws.kbarh, ws.vbarh, ws.vt, s.N,
                                                                      s.NK, s.NKr, s.NC, routing ? 1 : 0);
        else
            prep_kv_kernel<64><<<dim3(nj, s.BH), dim3(256), 0, st>>>(kk, vv, ws.kbar, ws.kbarh, ws.vbarh, ws.vt, s.N,
                                                                     s.NK, s.NKr, s.NC, routing ? 1 : 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (routing) {
            if ((e = launch_pool_mean(q, ws.qbar, kBF16, s.BH, s.N, d, s.bq, st)) != hipSuccess) return e;
            if (!s.causal) {   // causal masks: the kernel takes each row's statistics itself
                if ((e = launch_moments(ws.kbar, ws.muk, ws.cov, ws.mom, s.BH, s.NK, s.NKr, d, st)) != hipSuccess)
                    return e;
                if ((e = launch_tau(ws.qbar, ws.muk, ws.cov, ws.tau, nullptr, ws.sigma, s.BH, s.NQ, d, beta, s.diag,
                                    st)) != hipSuccess)
                    return e;
                if ((e = launch_order(ws.qbar, ws.cov, ws.sigma, ws.order, s.BH, s.NQ, d, st)) != hipSuccess) return e;
            }
        }
        AttnArgs a{};
        a.order = (routing && !s.causal) ? ws.order : nullptr;
        a.queue = ws.queue;
        a.q = static_cast<const uint16_t*>(q);
        a.k = kk;
        a.vt = ws.vt;
        a.qbar = ws.qbar;
        a.kbar = ws.kbar;
        a.kbarh = ws.kbarh;
        a.vbarh = ws.vbarh;
        a.tau = ws.tau;
        a.out = static_cast<uint16_t*>(out);
        a.blkcount = ws.blkcount;
        a.mask_out = mask_out;
        a.BH = s.BH; a.N = s.N; a.NQ = s.NQ; a.NK = s.NK; a.NKr = s.NKr; a.NC = s.NC; a.MW = s.MW;
        a.hlog = s.causal ? 0 : heads_in_flight_log2(s);
        a.per_x = s.causal ? 2 * ((s.NQ + 15) / 16) : (s.NQ + (8 >> a.hlog) - 1) / (8 >> a.hlog);
        a.scale = scale;
        a.causal_g = s.causal;
        a.beta = beta;
        a.c_log2 = scale * kLog2e;
        a.bias_full = log2f((float)kBlockK) / a.c_log2;
        a.bias_last = log2f((float)(s.N - (s.NK - 1) * kBlockK)) / a.c_log2;
        queue_reset_kernel<<<1, 64, 0, st>>>(ws.queue);   // a fill kernel, not a memset: safe under graph capture
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (ev_start && (e = hipEventRecord(ev_start, st)) != hipSuccess) return e;
        if (d == 128) e = s.bq == 128 ? dispatch_bf16<128, 128>(s, a, st) : dispatch_bf16<128, 64>(s, a, st);
        else e = s.bq == 128 ? dispatch_bf16<64, 128>(s, a, st) : dispatch_bf16<64, 64>(s, a, st);
        if (e != hipSuccess) return e;
        if (ev_stop && (e = hipEventRecord(ev_stop, st)) != hipSuccess) return e;
    } else {
        if (routing) {
            if ((e = launch_pool_mean(q, ws.qbar, kF32, s.BH, s.N, d, s.bq, st)) != hipSuccess) return e;
            if ((e = launch_pool_mean(k, ws.kbar, kF32, s.BH, s.N, d, s.bk, st)) != hipSuccess) return e;
            if (s.mode == kSparse && (e = launch_pool_mean(v, ws.vbar, kF32, s.BH, s.N, d, s.bk, st)) != hipSuccess)
                return e;
            if (!s.causal) {
                if ((e = launch_moments(ws.kbar, ws.muk, ws.cov, ws.mom, s.BH, s.NK, s.NKr, d, st)) != hipSuccess)
                    return e;
                if ((e = launch_tau(ws.qbar, ws.muk, ws.cov, ws.tau, nullptr, nullptr, s.BH, s.NQ, d, beta, s.diag,
                                    st)) != hipSuccess)
                    return e;
            }
        }
        AttnArgsF32 a{};
        a.q = static_cast<const float*>(q);
        a.k = static_cast<const float*>(k);
        a.v = static_cast<const float*>(v);
        a.qbar = ws.qbar;
        a.kbar = ws.kbar;
        a.vbar = ws.vbar;
        a.tau = ws.tau;
        a.out = static_cast<float*>(out);
        a.blkcount = ws.blkcount;
        a.mask_out = mask_out;
        a.BH = s.BH; a.N = s.N; a.NQ = s.NQ; a.NK = s.NK; a.NKr = s.NKr; a.NC = s.NC; a.MW = s.MW;
        a.scale = scale;
        a.causal_g = s.causal;
        a.beta = beta;
        if (ev_start && (e = hipEventRecord(ev_start, st)) != hipSuccess) return e;
        if (d == 128) e = s.bq == 128 ? dispatch_f32<128, 128>(s, a, st) : dispatch_f32<128, 64>(s, a, st);
        else e = s.bq == 128 ? dispatch_f32<64, 128>(s, a, st) : dispatch_f32<64, 64>(s, a, st);
        if (e != hipSuccess) return e;
        if (ev_stop && (e = hipEventRecord(ev_stop, st)) != hipSuccess) return e;
    }
    count_reduce_kernel<<<dim3(s.BH), dim3(256), 0, st>>>(ws.blkcount, counts, s.NQ);
    return hipGetLastError();
}

}  // namespace sol
