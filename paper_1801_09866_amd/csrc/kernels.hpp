// Kernel launchers shared between the HIP translation units and the C ABI.
#pragma once

#include <hip/hip_ext.h>

#include "common.hpp"

namespace rn {

// Optional timestamps of a stage: the dispatch packet of its first kernel
// stamps `start` when that kernel begins, the last kernel's stamps `stop` when
// it ends (hipExtLaunchKernel), so the elapsed time is kernel execution only.
struct Stamp {
    hipEvent_t start = nullptr, stop = nullptr;
};

template <typename... KArgs, typename... Args>
inline void launch_k(void (*k)(KArgs...), unsigned grid, unsigned block, hipStream_t s, Stamp ts, Args... args) {
    hipExtLaunchKernelGGL(k, dim3(grid), dim3(block), 0, s, ts.start, ts.stop, 0, args...);
}

void launch_fill_u32(void *p, uint32_t v, long long n, hipStream_t s);
void launch_fold_stats(const Dev &d, const FoldParts &fp, hipStream_t s);
// The launches of one frame block (one frame per session, fb.n of them).
void launch_hist_key(const Dev &d, const FrameBlock &fb, const DecadeTab &T, hipStream_t s, Stamp ts = {});
void launch_frame_plan(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts = {});
void launch_score_finish(const Dev &d, const FrameBlock &fb, hipStream_t s, Stamp ts = {});
void launch_debug_quantize(const float *x, long long n, int qmode, int k, const DecadeTab &T,
                           void *codes, int *err, hipStream_t s);

// GRU step for the work lists of all the block's frames, one launch per layer
// (max_rows bounds the device-side total row count).
void launch_gru_layer(const Dev &d, const FrameBlock &fb, int layer, int max_rows, hipStream_t s, Stamp ts = {});
// concatenate W_ih | W_hh of one layer into the packed [3H][Kx+H] layout
void launch_pack_layer(const Dev &d, int layer, const void *W_ih, const void *W_hh, void *dst,
                       hipStream_t s);


int lognorm_tiles(int V);
// The allocation-free normaliser keeps its partial pairs in a static device
// array sized for kStaticMaxTiles vocabulary tiles (256 rows per launch);
// its address on the current device (looked up once per device).
constexpr int kStaticMaxTiles = 2048;
constexpr int kStaticMaxV = kStaticMaxTiles * 208;   // vocabulary tiles of 208 words
constexpr int kMaxDevices = 64;
hipError_t lognorm_static_scratch(float2 **ptr);
// words: optional [n][3] context words; when given, the MaxEnt weights of
// every vocabulary word after each row's context join its logit
void launch_lognorm_gemm(const Dev &d, const float *h, const int32_t *words, int n, hipStream_t s, Stamp ts = {});
void launch_lognorm_combine(const Dev &d, int n, float *logz, hipStream_t s, Stamp ts = {});

}  // namespace rn
