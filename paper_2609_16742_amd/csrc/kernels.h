// Internal launcher interface between the host runtime and the gfx950
// kernels.  Not part of the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ctc {

enum DT { DT_F32 = 0, DT_F16 = 1 };

// Optional timing of the next kernel launch on this thread: when both
// events are set, the launcher dispatches with hipExtLaunchKernelGGL so the
// events carry the kernel's own start / end timestamps; cleared after use.
void set_launch_events(hipEvent_t start, hipEvent_t stop);
// True while events set by set_launch_events have not been used yet.
bool launch_events_pending();

struct ConvArgs {
    const void *x;        // [nimg][H][W][Cs]
    const void *w;        // [N][R][S][Cs]  (depthwise: [R][S][N])
    const float *scale;   // [N]
    const float *shift;   // [N]
    const void *res;      // [nimg][P][Q][N] or null
    void *y;              // [nimg][P][Q][N]
    int nimg, H, W, Cs, P, Q, N, R, S, stride, pad, relu;
};

// Dense (groups == 1) implicit-GEMM convolution on MFMA.
hipError_t launch_conv(int dt, const ConvArgs &a, hipStream_t st);
// Spatial-tile convolution for layers with few channels: one workgroup per
// (image, TH x TW output tile, 16*IN output channels); the input patch and
// the weights of a 16-byte channel chunk are staged in LDS once and every
// tap reads its shifted window from there.
struct TileCfg {
    int TH, TW;      // output tile
    int IMW;         // 16-pixel MFMA tiles per wave (tile has <= 64*IMW px)
    int IN;          // 16-channel MFMA tiles per workgroup
    int KS;          // kernel size (1 or 3)
};
// Tile choice for a conv (IMW == 0: use the implicit-GEMM kernel).
TileCfg choose_tile(int dt, const ConvArgs &a);
hipError_t launch_conv_tile(int dt, const ConvArgs &a, const TileCfg &c,
                            hipStream_t st);
const char *conv_tile_name(int dt, const TileCfg &c);

// Short name of the conv_igemm instance launch_conv picks for these args.
const char *conv_kernel_name(int dt, const ConvArgs &a);
// Depthwise convolution (direct, no MFMA).
hipError_t launch_dwconv(int dt, const ConvArgs &a, hipStream_t st);

hipError_t launch_maxpool(int dt, const void *x, void *y, int nimg, int H,
                          int W, int C, int P, int Q, int k, int stride,
                          int pad, hipStream_t st);
hipError_t launch_gap(int dt, const void *x, void *y, int nimg, int HW,
                      int C, hipStream_t st);

struct FcArgs {
    const void *x;        // [nimg][I]
    const void *w;        // [O][I]
    const float *shift;   // [O]
    void *y;              // rows < nmain: y + r*ld; else y2 + map2[r-nmain]*ld
    void *y2;
    const int32_t *map2;
    int nimg, nmain, I, O, ld, relu;
};
// dt_in / dt_w / dt_out in {DT_F32, DT_F16}
hipError_t launch_fc(int dt_in, int dt_w, int dt_out, const FcArgs &a,
                     hipStream_t st);

// NCHW fp32 -> NHWC (Cs channels, zero padded) in dt; images b >= nb are
// copied from `pend` (already staged, [npend][H][W][Cs]).
hipError_t launch_stage(int dt, const float *x, int nb, int C, int H, int W,
                        int Cs, void *t0, int npend, const void *pend,
                        hipStream_t st);

// Detector: flags[i] = !(|S_i - ref| <= tau), *count and the ascending
// indices of flagged rows in idx (either may be null); then (if pend !=
// null) copies the staged input of every flagged image into pend
// (img_bytes each).
hipError_t launch_verify(const float *out, int nb, int ld, int col, float ref,
                         float tau, uint8_t *flags, int32_t *count,
                         int32_t *idx, const void *src, void *pend,
                         size_t img_bytes, hipStream_t st);

struct ActFault {
    int64_t offset;  // byte offset within one image
    int32_t image;
    int32_t bit;
    int32_t width;   // 16 or 32
    int32_t pad_;
};
hipError_t launch_act_faults(void *base, size_t img_bytes, const ActFault *f,
                             int n, int nimg, hipStream_t st);
// Stores `bits` (16 or 32 wide) at a device address.
hipError_t launch_set_bits(void *addr, uint32_t bits, int width,
                           hipStream_t st);

}  // namespace ctc
