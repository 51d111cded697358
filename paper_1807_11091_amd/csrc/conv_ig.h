// Host interface of the implicit-GEMM CONV kernel for conv groups whose
// compacted columns are every tap times one run of consecutive input channels
// (conv_ig.hip).  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "sa_device.h"
#include "structadmm.h"

namespace sa {

// One conv group of a launch (every group of a layer runs in one launch).
struct IgGroup {
    const uint16_t *Wc;  // the group's compacted matrix [M][ldk], tap-major columns
    int32_t M, K, ldk;   // kept filters, kept columns (= taps * run), row pitch (multiple of 64)
    int32_t run;         // consecutive input channels per tap (multiple of 8)
    int32_t run_base;    // first input channel of the run (multiple of 8)
    int32_t o_off;       // first output channel of the group
    int32_t mtiles, begin;  // filled by the launcher
    FastDiv divRun;
};

struct IgArgs {
    const uint16_t *X;  // bf16 NHWC [N, H, W, Cx], 16-byte aligned
    uint16_t *Y;        // bf16 NHWC rows of ldy >= Cy elements, 4-byte aligned
    uint32_t x_bytes;
    int32_t yshift;     // elements from the 16-byte boundary below Y to Y
    int32_t H, W, Cx, D, stride, pad, P, Q, NPQ, Cy, ldy;
    int32_t ngroups, ntiles;
    FastDiv divPQ, divQ, divD, divCy;
    IgGroup g[SA_MAX_CONV_GROUPS];
};

// Tile shape the launcher takes for these groups (index into its table).
int ig_pick(const IgArgs &a);
// Number of tile shapes the launcher has, and the shape of tile t.
int ig_num_tiles();
void ig_tile_shape(int t, int *MT, int *NF, int *WM);
// Compute units of the current device (256 when it cannot be asked).
int device_cus();
// Launches every group of a (tile < 0: ig_pick's choice).
int ig_run(IgArgs a, int tile, hipStream_t stream);

}  // namespace sa
