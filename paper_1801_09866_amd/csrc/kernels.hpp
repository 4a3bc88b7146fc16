// Kernel launchers shared between the HIP translation units and the C ABI.
#pragma once

#include "common.hpp"

namespace rn {

void launch_fill_u32(void *p, uint32_t v, long long n, hipStream_t s);
void launch_fold_stats(const Dev &d, int npart, hipStream_t s);
void launch_hist_key(const Dev &d, const FrameArgs &f, const DecadeTab &T, hipStream_t s);
void launch_frame_plan(const Dev &d, const FrameArgs &f, int npart, hipStream_t s);
void launch_score_finish(const Dev &d, const FrameArgs &f, hipStream_t s);
void launch_debug_quantize(const float *x, long long n, int qmode, int k, const DecadeTab &T,
                           void *codes, int *err, hipStream_t s);

// GRU step for the frame's work list, one launch per layer (max_rows bounds
// the device-side row count).
void launch_gru_layer(const Dev &d, const FrameArgs &f, int layer, int max_rows, hipStream_t s);
// concatenate W_ih | W_hh of one layer into the packed [3H][Kx+H] layout
void launch_pack_layer(const Dev &d, int layer, const void *W_ih, const void *W_hh, void *dst,
                       hipStream_t s);


int lognorm_tiles(int V);
void launch_lognorm_gemm(const Dev &d, const float *h, int n, hipStream_t s);
void launch_lognorm_combine(const Dev &d, int n, float *logz, hipStream_t s);

}  // namespace rn
