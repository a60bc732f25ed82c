// Internal interface between the C ABI (sol_attn_api.cpp) and the gfx950
// kernels (sol_attn_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace sol {

constexpr int kBlockK = 64;        // key block size (rows of one exact K/V tile)
constexpr int kChunk = 64;         // pooled keys per correction tile
constexpr int kMaxLds = 160 * 1024;

enum Mode { kDense = 0, kSparse = 1, kSparseNoCorr = 2 };
constexpr int kThresholdDiagonal = 0x100;   // flag bit of the ABI mode (SOL_THRESHOLD_DIAGONAL)
enum DType { kBF16 = 0, kF32 = 1 };

// Derived sizes of one forward call.
struct Shape {
    int B, H, N, d, bq, bk;
    int mode, dtype, forced;       // forced = number of always-exact tail key blocks
    int diag;                      // 1: diagonal threshold estimator
    int causal;                    // causal granule G (0: no mask); key s visible to query t iff
                                   // s < min((t / G + 1) G, N)
    int BH, NQ, NK, NKr, NC, Npad, MW;
};

// `mode` is the ABI mode: base mode plus optional kThresholdDiagonal.
Shape make_shape(int B, int H, int N, int d, int bq, int bk, int mode, int dtype, int keep_tail_tokens,
                 int causal_granule = 0);

// Workspace carve-up (all device pointers, 256-byte aligned inside one buffer).
struct Workspace {
    float* qbar = nullptr;       // [BH][NQ][d]
    float* kbar = nullptr;       // [BH][NK][d]
    float* vbar = nullptr;       // [BH][NK][d]            (f32 path)
    _Float16* kbarh = nullptr;   // [BH][NC*64][d] f16      (bf16 routing modes)
    _Float16* vbarh = nullptr;   // [BH][NC*64][d] f16      (bf16 sparse)
    _Float16* vt = nullptr;      // [BH][NK][d][64] f16     (bf16)
    float* muk = nullptr;        // [BH][d]
    float* cov = nullptr;        // [BH][d][d]
    float* tau = nullptr;        // [BH][NQ]
    float* sigma = nullptr;      // [BH][NQ] sigma_i of the thresholds (query-block order)
    uint16_t* order = nullptr;   // [BH][NQ] query-block order of the sparse kernels
    double* mom = nullptr;       // partial moments, moments_scratch_bytes()
    uint32_t* blkcount = nullptr;// [BH][NQ]
    uint32_t* queue = nullptr;   // [8][32] per-XCD claim counters of the bf16 attention kernel (one per 128 B)
};

// Returns the byte size; fills *ws when base != nullptr.
size_t workspace_layout(const Shape& s, char* base, Workspace* ws);

// Dynamic LDS bytes of the fused attention kernel for this shape.
size_t attn_lds_bytes(const Shape& s);

hipError_t launch_pool_mean(const void* x, float* mean, int dtype, int BH, int N, int d, int blk,
                            hipStream_t st);
size_t moments_scratch_bytes(int BH, int NKr, int d);
hipError_t launch_moments_final(const float* kbar, float* muk, float* cov, double* scratch, int BH, int NK, int NKr,
                                int d, hipStream_t st);
hipError_t launch_moments(const float* kbar, float* muk, float* cov, double* scratch, int BH, int NK, int NKr,
                          int d, hipStream_t st);
hipError_t launch_tau(const float* qbar, const float* muk, const float* cov, float* tau, float* mu,
                      float* sigma, int BH, int NQ, int d, float beta, int diag, hipStream_t st);
// Materialised-proxy routing baselines (top-k: rule 0, param = k; top-p: rule 1, param = p).
hipError_t launch_route_materialized(const float* qbar, const float* kbar, float* shat, uint32_t* mask, int BH, int NQ,
                                     int NK, int NKr, int d, int rule, float param, hipStream_t st);
// Built-in device scratch of the entry point that allocates nothing (one array per device in the
// code object): its size, and its device address on the current device (looked up once per
// device with hipGetSymbolAddress).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(void** addr);

// ev_start/ev_stop (nullable) are recorded on `st` around the fused attention kernel.
hipError_t launch_forward(const Shape& s, const void* q, const void* k, const void* v, void* out,
                          float beta, const Workspace& ws, uint32_t* counts, uint32_t* mask_out,
                          hipStream_t st, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

}  // namespace sol
