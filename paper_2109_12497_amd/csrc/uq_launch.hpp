// Launch planning shared by the kernels and the ABI layer of libuq.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "uq_device.hpp"

namespace uq {

// The norm's reduction tree: chunks of `chunk` coordinates (a multiple of
// 8192, so every chunk starts 16-byte aligned), at most 1024 chunks per row.
// It depends on d only, which makes W independent of the device and of the
// launch geometry.
struct NormPlan {
    int64_t chunk;
    int32_t nchunks;
};

inline NormPlan norm_plan(int64_t d)
{
    const int64_t base = 8192;
    const int64_t per = base * 1024;
    const int64_t mult = d > 0 ? (d + per - 1) / per : 1;
    NormPlan p;
    p.chunk = base * mult;
    p.nchunks = static_cast<int32_t>(d > 0 ? (d + p.chunk - 1) / p.chunk : 0);
    return p;
}

// Several scales and 2 to kFuseRows rows: one pass over the gradients
// yields both the rows' sums of squares and the largest |g| over the rows at
// every coordinate (the input of the scale index), so the gradients are read
// once instead of twice.  Its reduction tree depends on d only: one fp64
// partial per row and tile of kFusedTile coordinates (whole quads) and one
// for the d % 4 trailing coordinates, then fixed-order sums of kRowsumSpan
// consecutive partials, then of those.
constexpr int32_t kFuseRows = 16;
constexpr int64_t kFusedTile = 1024;
constexpr int64_t kRowsumSpan = 16384;

struct FusedPlan {
    int64_t ntiles;  // tiles of kFusedTile coordinates in whole quads (the last one may be partial)
    int64_t nsub;    // sums of kRowsumSpan consecutive partials (ntiles + 1 per row)
};

inline FusedPlan fused_plan(int64_t d)
{
    FusedPlan p;
    const int64_t nquad = d > 0 ? d / 4 : 0;
    p.ntiles = (nquad + kFusedTile / 4 - 1) / (kFusedTile / 4);
    p.nsub = (p.ntiles + 1 + kRowsumSpan - 1) / kRowsumSpan;
    return p;
}

// The index pass's constants for one call, formed once from the rows' sums
// (k_index_prep) instead of in every block of the pass: each scale's
// threshold T_k and its 16-bit key, the 256-entry exponent table, and
// whether that table decides every key (no binade holds two thresholds).
struct IndexTables {
    uint2 tab[256];
    float thr[kMaxScales];
    uint32_t hk[kMaxScales];
    int32_t by_table;
};

// Workspace of the fused path, in bytes from the start of the workspace:
// tile partials [M][ntiles + 1] fp64, their sums [M][nsub] fp64, row sums
// [M] fp64, the index pass's IndexTables, then, from the first 4 KiB
// boundary of the address at or after keys_off (fused_keys), the row
// maxima's 16-bit keys [d] followed by one spare quad (padding; nothing is
// stored there).  A block of the norm pass stores the keys of 1024
// coordinates, 2 KiB, so with the keys 4 KiB aligned each store fills
// aligned 2 KiB.  Measured on MI355X at 2^30 coordinates and 16 rows, in a
// work-free probe of the pass's access pattern: key buffers at multiples of
// 1024 bytes ran up to 2.5% faster than at other multiples of 256.  (The
// pass's time also depends on where the gradients lie in memory: 11.2 to
// 12.5 ms on different boxes with these keys.)
constexpr size_t kKeysAlign = 4096;

struct FusedLayout {
    size_t sub_off;
    size_t rows_off;
    size_t tab_off;
    size_t keys_off;
    size_t bytes;
};

inline size_t align256(size_t n)
{
    return (n + 255) / 256 * 256;
}

inline FusedLayout fused_layout(int64_t d, int32_t M)
{
    const FusedPlan p = fused_plan(d);
    FusedLayout L;
    L.sub_off = align256(static_cast<size_t>(M) * static_cast<size_t>(p.ntiles + 1) * sizeof(double));
    L.rows_off = L.sub_off + align256(static_cast<size_t>(M) * static_cast<size_t>(p.nsub) * sizeof(double));
    L.tab_off = L.rows_off + align256(static_cast<size_t>(M) * sizeof(double));
    L.keys_off = L.tab_off + align256(sizeof(IndexTables));
    L.bytes = L.keys_off + kKeysAlign + align256(static_cast<size_t>((d + 3) / 4 * 4 + 4) * sizeof(uint16_t));
    return L;
}

// The keys' start in the workspace ws (any 16-byte aligned address).
inline uint16_t* fused_keys(void* ws, const FusedLayout& L)
{
    const uintptr_t p = reinterpret_cast<uintptr_t>(ws) + L.keys_off;
    return reinterpret_cast<uint16_t*>((p + kKeysAlign - 1) / kKeysAlign * kKeysAlign);
}

// One row gains nothing: the fused pass then moves more bytes (13 per
// coordinate against 9) and measured slower.
inline bool use_fused(int64_t d, int32_t M, int32_t K)
{
    return K > 1 && d > 0 && M >= 2 && M <= kFuseRows;
}

// Upper bound on blocks for the grid-stride kernels: 64 blocks of 256
// threads per compute unit of the current device.
int64_t grid_cap();

// The cap on the one-shot grids of the streaming passes (norm, index,
// quantise, sum, reconstruction): 2^22 blocks unless lowered, to no fewer than
// kMinOneShotCap, by the test hook.  Returns false for a value out of range.
constexpr int64_t kMinOneShotCap = 8;
bool set_one_shot_cap(int64_t blocks);

// ws: at least uq_workspace_bytes(d, M) bytes (norm partials, or the fused
// path's layout); idx_bits as for launch_quant_sum
hipError_t launch_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, const ScaleSet& S,
                               float* w, uint8_t* idx, void* ws, hipStream_t stream, int32_t idx_bits = 8);
// bits = 8: int8 codes [rows][ldc]; bits = 4 or 2: packed codes, ldc in bytes
hipError_t launch_quantise(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                           const float* w, const ScaleSet& S, const uint8_t* idx, uint64_t seed,
                           void* codes, int64_t ldc, int32_t bits, hipStream_t stream);
// quantise `rows` rows and add their codes into sum (= or +=) without storing
// them; out != nullptr: also the reconstruction of the stored sums (M workers);
// idx_bits 8: one byte per coordinate, 4: two coordinates a byte (low nibble
// first)
hipError_t launch_quant_sum(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                            const ScaleSet& S, const uint8_t* idx, uint64_t seed, int32_t accumulate, int32_t* sum,
                            int32_t M, float* out, hipStream_t stream, int32_t idx_bits = 8);
hipError_t launch_index_quant_sum(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                                  const ScaleSet& S, uint64_t seed, uint8_t* idx, int32_t* sum, float* out,
                                  hipStream_t stream);
// several scales, M <= 16 rows: the shared index formed from the rows'
// maxima (stored to idx) and every row's codes stored (bits 8, 4 or 2)
hipError_t launch_index_quantise(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                                 const ScaleSet& S, uint64_t seed, int32_t bits, uint8_t* idx, uint8_t* codes,
                                 int64_t ldc, hipStream_t stream);
hipError_t launch_sum_packed(const uint8_t* packed, int64_t d, int32_t rows, int64_t ldp, int32_t bits,
                             int32_t accumulate, int32_t* sum, hipStream_t stream);
hipError_t launch_sum(const int8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t accumulate,
                      int32_t* sum, hipStream_t stream);
// the sum (bits = 8, 4 or 2) with the reconstruction applied to the sums it stores
hipError_t launch_sum_dequant(const uint8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t bits,
                              int32_t accumulate, int32_t* sum, int32_t M, const float* w, const ScaleSet& S,
                              const uint8_t* idx, float* out, hipStream_t stream);
// GlobalRandK: at most kRandkCandidates keys sharing the threshold's 20-bit
// prefix are kept (expected d / 2^20 <= 4096 for d < 2^32, standard deviation
// 64 at most); when more arrive, an exact refinement finds the threshold.
constexpr int kRandkCandidates = 8192;

size_t randk_workspace_bytes();
// How the K-subset is found (test hook): the bracket with its exact
// fallback (default), the multi-pass histograms, or the bracket made to miss.
// The two NoCandidates modes keep no boundary candidates, so that the exact
// refinement always runs (histogram route, and the bracket's fallback).
constexpr int32_t kRandkBracket = 1, kRandkHistogram = 0, kRandkBracketMiss = 2;
constexpr int32_t kRandkHistogramNoCandidates = 3, kRandkBracketMissNoCandidates = 4;
bool set_randk_mode(int32_t mode);
hipError_t launch_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* sel, void* ws, hipStream_t stream);
hipError_t launch_gather(const float* g, int64_t d, int32_t M, int64_t ldg, const uint32_t* sel, int64_t K,
                         float* sub, int64_t lds, hipStream_t stream);
hipError_t launch_scatter(const float* vals, const uint32_t* sel, int64_t K, float* out, int64_t d,
                          hipStream_t stream);
hipError_t launch_dequant(const int32_t* sum, int64_t d, int32_t M, const float* w, const ScaleSet& S,
                          const uint8_t* idx, float* out, hipStream_t stream);

}  // namespace uq
