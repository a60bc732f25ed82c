// Routing baselines with a materialised proxy map (the standard routing the paper compares
// against, Section 2 after Eq. block_proxy): the full proxy map s_hat = s * Qbar Kbar^T is
// written to memory, then every row is traversed again by a top-k or a top-p rule.  These
// kernels exist to measure what on-the-fly routing avoids; the forward pass never uses them.
//
//   proxy_map_kernel   s_hat[bh][i][j], f32, 64 x 64 output tiles
//   topk_kernel        k largest proxies of a row: radix select on order-preserving keys,
//                      ties to the lower key-block index
//   topp_kernel        shortest decreasing prefix of Softmax(s_hat_i) with mass >= p: bitonic
//                      sort of the row in LDS, then an exclusive prefix sum of the weights
#include "sol_attn_internal.h"

#include <cmath>

namespace sol {
namespace {

// Order-preserving map of a float to an unsigned key (larger float -> larger key).
__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// ---------------------------------------------------------------------------
// s_hat[bh][i][j] = scale * Qbar[bh][i] . Kbar[bh][j], j < NKr.  grid (ceil(NKr/64),
// ceil(NQ/64), BH), 256 threads; thread t owns rows 4*(t/16).. and columns 4*(t%16)..
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void proxy_map_kernel(const float* __restrict__ qbar, const float* __restrict__ kbar,
                                                        float* __restrict__ shat, int NQ, int NK, int NKr, float scale) {
    constexpr int DC = 32;   // d columns staged per step
    __shared__ float qs[64][DC + 1];
    __shared__ float ks[64][DC + 1];
    const int j0 = blockIdx.x * 64, i0 = blockIdx.y * 64, bh = blockIdx.z, t = threadIdx.x;
    const int ti = (t / 16) * 4, tj = (t % 16) * 4;
    float acc[4][4] = {};
    for (int c0 = 0; c0 < D; c0 += DC) {
        for (int e = t; e < 64 * DC; e += 256) {
            const int r = e / DC, c = e % DC;
            const int i = min(i0 + r, NQ - 1), j = min(j0 + r, NKr - 1);
            qs[r][c] = qbar[((size_t)bh * NQ + i) * D + c0 + c];
            ks[r][c] = kbar[((size_t)bh * NK + j) * D + c0 + c];
        }
        __syncthreads();
#pragma unroll 8
        for (int c = 0; c < DC; ++c) {
            float a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a[u] = qs[ti + u][c];
                b[u] = ks[tj + u][c];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[u][v] = fmaf(a[u], b[v], acc[u][v]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int i = i0 + ti + u, j = j0 + tj + v;
            if (i < NQ && j < NKr) shat[((size_t)bh * NQ + i) * NKr + j] = scale * acc[u][v];
        }
}

// ---------------------------------------------------------------------------
// Top-k of each row.  grid (NQ, BH), 256 threads, NKr <= 8192; the row's keys are staged
// in LDS (dynamic, NKr u32).  Radix select, 8 bits per pass from the top, finds the key K of the
// k-th largest proxy; keys above K are kept, and of the keys equal to K the lowest indices
// until k are kept.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ shat, uint32_t* __restrict__ mask, int NQ,
                                                   int NKr, int MW, int k) {
    extern __shared__ uint32_t keys[];
    __shared__ int hist[256];
    __shared__ int scratch[8];
    __shared__ uint32_t prefix_s;
    __shared__ int need_s;
    const int i = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
    const float* row = shat + ((size_t)bh * NQ + i) * NKr;
    for (int j = t; j < NKr; j += 256) keys[j] = order_key(row[j]);
    if (t == 0) {
        prefix_s = 0u;
        need_s = k;
    }
    __syncthreads();
    // radix select: at each pass the keys matching the prefix so far are counted by digit
    for (int shift = 24; shift >= 0; shift -= 8) {
        hist[t] = 0;
        __syncthreads();
        const uint32_t prefix = prefix_s;
        const uint32_t hmask = shift == 24 ? 0u : (0xFFFFFFFFu << (shift + 8));
        for (int j = t; j < NKr; j += 256) {
            const uint32_t key = keys[j];
            if ((key & hmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        __syncthreads();
        if (t == 0) {
            int need = need_s, dgt = 255;
            for (; dgt > 0; --dgt) {
                if (hist[dgt] >= need) break;
                need -= hist[dgt];
            }
            prefix_s = prefix | ((uint32_t)dgt << shift);
            need_s = need;
        }
        __syncthreads();
    }
    const uint32_t kth = prefix_s;   // key of the k-th largest proxy
    const int take_eq = need_s;      // how many of the keys equal to kth are kept
    // keep: key > kth, or key == kth among the first take_eq such indices.  Thread t owns mask
    // word t (MW <= 256); an exclusive scan of the per-word counts of keys equal to kth gives
    // each word the number of equal keys before it.
    const int w = t;
    int eq_in_word = 0;
    if (w < MW)
        for (int b = 0; b < 32 && w * 32 + b < NKr; ++b) eq_in_word += keys[w * 32 + b] == kth;
    int incl = eq_in_word;
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off);
        if ((t & 63) >= off) incl += y;
    }
    if ((t & 63) == 63) scratch[t >> 6] = incl;
    __syncthreads();
    int seen = incl - eq_in_word;
    for (int u = 0; u < (t >> 6); ++u) seen += scratch[u];
    if (w < MW) {
        uint32_t bits = 0;
        for (int b = 0; b < 32 && w * 32 + b < NKr; ++b) {
            const uint32_t key = keys[w * 32 + b];
            if (key > kth) {
                bits |= 1u << b;
            } else if (key == kth) {
                if (seen < take_eq) bits |= 1u << b;
                ++seen;
            }
        }
        mask[((size_t)bh * NQ + i) * MW + w] = bits;
    }
}

// ---------------------------------------------------------------------------
// Top-p of each row.  grid (NQ, BH), 256 threads; NP = next power of two >= NKr (<= 4096)
// entries of (key << 32 | ~index) sorted in decreasing order in LDS (bitonic), so equal
// proxies come in increasing index order; padding entries are 0 and sort last.  The
// weights exp(s - s_max) are then prefix-summed in sorted order, and entry t is kept when
// the mass before it is below p times the total.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void topp_kernel(const float* __restrict__ shat, uint32_t* __restrict__ mask, int NQ,
                                                   int NKr, int MW, int NP, float p) {
    extern __shared__ unsigned long long ent[];   // NP entries, then NP floats of weights
    float* wts = reinterpret_cast<float*>(ent + NP);
    __shared__ float part[256];
    __shared__ uint32_t mbits[128];               // MW <= 128
    const int i = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
    const float* row = shat + ((size_t)bh * NQ + i) * NKr;
    for (int j = t; j < NP; j += 256)
        ent[j] = j < NKr ? ((unsigned long long)order_key(row[j]) << 32) | (uint32_t)~(uint32_t)j : 0ull;
    for (int w = t; w < MW; w += 256) mbits[w] = 0u;
    __syncthreads();
    // bitonic sort, decreasing
    for (int size = 2; size <= NP; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int x = t; x < NP / 2; x += 256) {
                const int lo = 2 * x - (x & (stride - 1));
                const int hi = lo + stride;
                const bool desc = (lo & size) == 0;
                const unsigned long long a = ent[lo], b = ent[hi];
                if ((a < b) == desc) {
                    ent[lo] = b;
                    ent[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    // weights in sorted order, relative to the largest proxy
    const float smax = row[(int)~(uint32_t)(ent[0] & 0xFFFFFFFFull)];
    for (int x = t; x < NP; x += 256) {
        float wv = 0.f;
        if (x < NKr) wv = __expf(row[(int)~(uint32_t)(ent[x] & 0xFFFFFFFFull)] - smax);
        wts[x] = wv;
    }
    __syncthreads();
    // exclusive prefix sum over NP entries: each thread sums a contiguous run
    const int run = NP / 256 > 0 ? NP / 256 : 1;
    const int r0 = t * run;
    float local = 0.f;
    for (int x = r0; x < r0 + run && x < NP; ++x) local += wts[x];
    part[t] = local;
    __syncthreads();
    if (t == 0) {   // scan of the 256 partial sums (tiny)
        float acc = 0.f;
        for (int u = 0; u < 256; ++u) {
            const float v = part[u];
            part[u] = acc;
            acc += v;
        }
        wts[NP] = acc;   // total (the weights array has one spare slot: see the LDS size)
    }
    __syncthreads();
    const float limit = p * wts[NP];
    float before = part[t];
    for (int x = r0; x < r0 + run && x < NKr; ++x) {
        if (before < limit) {
            const int j = (int)~(uint32_t)(ent[x] & 0xFFFFFFFFull);
            atomicOr(&mbits[j >> 5], 1u << (j & 31));
        }
        before += wts[x];
    }
    __syncthreads();
    for (int w = t; w < MW; w += 256) mask[((size_t)bh * NQ + i) * MW + w] = mbits[w];
}

}  // namespace

hipError_t launch_route_materialized(const float* qbar, const float* kbar, float* shat, uint32_t* mask, int BH, int NQ,
                                     int NK, int NKr, int d, int rule, float param, hipStream_t st) {
    const float scale = 1.0f / sqrtf((float)d);
    const dim3 g((NKr + 63) / 64, (NQ + 63) / 64, BH);
    if (d == 128) proxy_map_kernel<128><<<g, dim3(256), 0, st>>>(qbar, kbar, shat, NQ, NK, NKr, scale);
    else proxy_map_kernel<64><<<g, dim3(256), 0, st>>>(qbar, kbar, shat, NQ, NK, NKr, scale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int MW = (NKr + 31) / 32;
    if (rule == 0) {
        const size_t lds = (size_t)NKr * 4;
        if (lds > 64 * 1024) {
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(topk_kernel),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
        }
        topk_kernel<<<dim3(NQ, BH), dim3(256), lds, st>>>(shat, mask, NQ, NKr, MW, (int)param);
    } else {
        int NP = 1;
        while (NP < NKr) NP <<= 1;
        if (NP < 512) NP = 512;
        const size_t lds = (size_t)NP * 8 + ((size_t)NP + 1) * 4;
        if (lds > 64 * 1024) {
            e = hipFuncSetAttribute(reinterpret_cast<const void*>(topp_kernel),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
        }
        topp_kernel<<<dim3(NQ, BH), dim3(256), lds, st>>>(shat, mask, NQ, NKr, MW, NP, param);
    }
    return hipGetLastError();
}

}  // namespace sol
