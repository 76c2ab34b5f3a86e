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
    // optional scratch for split-K layers: [conv_splitk()][nimg*P*Q][N]
    // fp32 partial sums (null: no split)
    float *part;
    int ksplit;           // set by launch_conv
    // 2: a 2x2 stride-2 max pool follows in the same kernel; y is then the
    // pooled map [nimg][P/2][Q/2][N] (0: no pool)
    int pool;
};
// Number of k ranges launch_conv splits this layer into when a.part is
// given (1: none).  Depends on the layer's shape, not on a.nimg, so every
// image's arithmetic is the same at any batch size.
int conv_splitk(int dt, const ConvArgs &a);

// Dense (groups == 1) implicit-GEMM convolution on MFMA.  With a.pool == 2
// the 2x2 stride-2 max pool after it runs in the conv's epilogue (only
// where conv_pool_ok; hipErrorInvalidValue else).
hipError_t launch_conv(int dt, const ConvArgs &a, hipStream_t st);
// Whether launch_conv can fuse the 2x2 / 2 max pool into this conv.
bool conv_pool_ok(int dt, const ConvArgs &a);
// Device address of the static scratch array (split-K partial sums of the
// allocation-free conv entry point) on the current device, looked up once
// per device; and its size in bytes.
hipError_t conv_scratch(void **ptr);
size_t conv_scratch_bytes();
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


// One row of a forward pass.  The host writes the table into pinned host
// memory; the pass's assemble kernel copies it to device memory, where the
// final FC and the detector read it.
struct RowEnt {
    int64_t out;     // device address of the row's output (logits, then S)
    int64_t flags;   // device address of its flag byte, or 0
    int32_t slot;    // ring slot holding its staged input, or -1
    int32_t first;   // 1: first execution (verified); 0: a re-execution
};

struct FcArgs {
    const void *x;        // [nimg][I]
    const void *w;        // [O][I]
    const float *shift;   // [O]
    void *y;              // row r at y + r*ld, unless rows is set:
    const RowEnt *rows;   //   then row r at rows[r].out (fp32 output)
    int nimg, I, O, ld, relu;
    // fused detector (Sec. II-B) on output det_col (-1: none), first
    // executions only: flag byte to rows[r].flags and flag_pass[r] (the
    // pass's own flag row in device memory, 0 for re-executions)
    int det_col;
    float ref, tau;
    uint8_t *flag_pass;
    // fp32 partial sums of the k ranges when fc_part_bytes() > 0
    float *part;
};

// Identity basic block in one kernel (fp32, C = 16, 32 or 64, both convs 3x3
// stride 1 pad 1, weights [C][3][3][C]):
// y = relu(conv2(relu(conv1(x) * sc1 + sh1)) * sc2 + sh2 + x), per TH x TW
// output tile, the conv1 result kept in LDS.
// Flag bytes of up to FLAG_SEGS passes from device memory (src[i], n[i]
// bytes) to pinned host memory (dst[i]), with system-scope stores.
constexpr int FLAG_SEGS = 4;
struct FlagCopy {
    const uint8_t *src[FLAG_SEGS];
    uint8_t *dst[FLAG_SEGS];
    int n[FLAG_SEGS];
    int nseg;
};
constexpr int BLOCK_STAGE_MAX = 128; // ring rows / extra conversions
struct BlockArgs {
    const void *x;                            // [nimg][H][W][C]
    const void *w1; const float *sc1, *sh1;
    const void *w2; const float *sc2, *sh2;
    void *y;                                  // [nimg][H][W][C]
    int nimg, H, W, C, TH, TW;
    // optional stem in front of the block (C = 16): x is then not read;
    // the block input is relu(conv3x3(x0) * sc0 + sh0), x0 [nimg][H][W][4],
    // w0 [16][3][3][4]
    const void *x0; const void *w0; const float *sc0, *sh0;
    // optional, with the stem: the pass input staged inside the kernel
    // instead of read from x0.  Rows below xs_n are the caller's images
    // xs[row] (xs: [xs_imgs][xs_c][H][W] fp32, xs_c <= 4); rows xs_n ..
    // nimg-1 (at most BLOCK_STAGE_MAX) are stored images in ring slots
    // rr_slot[] (ring: ring_bytes of [slot][H][W][4] fp32).  Every row is
    // also stored to x0 in x0's layout (channels past xs_c zero), which
    // later re-executions read.  ov_n more of the caller's images xs[ov_src[]]
    // are converted into ring slots ov_slot[] by ov_n extra workgroups.
    // nrows row-table entries are copied rows_host -> rows_dev, and the
    // flags of an earlier pass as `flags` says.
    const float *xs; int xs_c, xs_n, xs_imgs;
    const void *ring; long ring_bytes;
    int rr_slot[BLOCK_STAGE_MAX];
    int ov_n, ov_src[BLOCK_STAGE_MAX], ov_slot[BLOCK_STAGE_MAX];
    const RowEnt *rows_host; RowEnt *rows_dev; int nrows;
    FlagCopy flags;                           // by workgroup 0 (stem only)
    // optional head behind the block (C = 64): global average pooling of
    // each image and the small FC `fc` on it (fc.x unused; needs
    // gap_fc_ok(fc) and fc.O <= 16, fc.I == C), run by the last of the
    // image's workgroups to finish, with results bit-identical to
    // launch_gap_fc on y.  cnt: [nimg] arrival counters, zero before the
    // launch and left zero.
    bool head; FcArgs fc; int *cnt;
};
// kernel arguments are limited to 4 KB
static_assert(sizeof(BlockArgs) <= 3072, "BlockArgs too large for kernel arguments");
// Whether (C, TH, TW) is a compiled tile and the sizes fit.
bool block_ok(const BlockArgs &a);
// Sets a.TH / a.TW for a.nimg, a.H, a.W, a.C (0 when none applies).
void choose_block_tile(BlockArgs &a);
const char *block_kernel_name(const BlockArgs &a);
hipError_t launch_block(const BlockArgs &a, hipStream_t st);

// Downsampling basic block in one kernel (fp32, (Ci, Co) = (16, 32) or
// (32, 64)): y = relu(bn2(conv2(relu(bn1(conv1(x))))) + bns(convs(x)))
// with conv1 3x3 stride 2 pad 1 [Co][3][3][Ci], the shortcut convs 1x1
// stride 2 [Co][Ci], conv2 3x3 stride 1 pad 1 [Co][3][3][Co]; BN folded
// into scale / shift per output channel.
struct DownArgs {
    const void *x;                            // [nimg][H][W][Ci]
    const void *w1; const float *sc1, *sh1;
    const void *ws; const float *scs, *shs;
    const void *w2; const float *sc2, *sh2;
    void *y;                                  // [nimg][P][Q][Co]
    int nimg, H, W, P, Q, Ci, Co;
};
bool down_ok(const DownArgs &a);
long down_tiles(const DownArgs &a);           // workgroups of a launch
const char *down_kernel_name(const DownArgs &a);
hipError_t launch_down(const DownArgs &a, hipStream_t st);

// Short name of the conv_igemm instance launch_conv picks for these args.
const char *conv_kernel_name(int dt, const ConvArgs &a);
// Depthwise convolution (direct, no MFMA).
// MobileNetV2-type inverted residual block as one kernel: expand 1x1 (+BN,
// ReLU) -> depthwise 3x3 stride 1|2 pad 1 (+BN, ReLU) -> project 1x1 (+BN,
// optional residual, optional ReLU), fp16 tensors, the expanded tensors
// kept in LDS.  Weights as packed for the separate kernels: expand [E][C],
// depthwise [3][3][E], project [Co][E].
struct IrArgs {
    const void *x;                       // [nimg][H][W][C]
    const void *we; const float *sce, *she;
    const void *wd; const float *scd, *shd;
    const void *wp; const float *scp, *shp;
    const void *res;                     // [nimg][P][Q][Co] or null
    void *y;                             // [nimg][P][Q][Co]
    int nimg, H, W, C, E, Co, P, Q, stride, relu_p;
};
// Whether launch_ir handles these sizes (fp16; C % 8, E % 8, Co % 4;
// C <= 160, Co <= 320; stride 1 or 2).
bool ir_supported(const IrArgs &a);
// Whether launch_ir is faster than the separate kernels for this shape
// (fusion detection only fuses such blocks).
bool ir_profitable(const IrArgs &a);
const char *ir_kernel_name(const IrArgs &a);
hipError_t launch_ir(const IrArgs &a, hipStream_t st);
// Depthwise 3x3 (stride 1, pad 1) + BN (+ ReLU) -> pointwise 1x1 + BN
// (+ residual, + ReLU) in one fp16 kernel: an inverted-residual block
// without expansion (Sec. II-A's MobileNet blocks, expansion factor 1).
struct DwPwArgs {
    const void *x;                       // [nimg][H][W][C]
    const void *wd; const float *scd, *shd;   // depthwise [3][3][C]
    const void *wp; const float *scp, *shp;   // pointwise [Co][C]
    const void *res;                     // [nimg][H][W][Co] or null
    void *y;                             // [nimg][H][W][Co]
    int nimg, H, W, C, Co, relu_d, relu_p;
};
// Whether launch_dwpw handles these sizes (C % 8, C <= 32, Co % 4, Co <= 64)
// and is faster there than the two separate kernels.
bool dwpw_supported(const DwPwArgs &a);
hipError_t launch_dwpw(const DwPwArgs &a, hipStream_t st);
// Name of the depthwise kernel launch_dwconv picks for these arguments.
const char *dwconv_kernel_name(int dt, const ConvArgs &a);
hipError_t launch_dwconv(int dt, const ConvArgs &a, hipStream_t st);

// fp16 7x7 stride-2 stem conv (4 stored input channels, 32 or 64 outputs,
// BN + ReLU in scale / shift / relu) followed by a 3x3 stride-2 pad-1 max
// pool into y [nimg][PP][QP][N], in one kernel; bit-identical to
// launch_conv then launch_maxpool.
bool stem_pool_ok(int dt, const ConvArgs &a, int PP, int QP);
const char *stem_pool_kernel_name(const ConvArgs &a);
hipError_t launch_stem_pool(const ConvArgs &a, int PP, int QP, hipStream_t st);

// Name of the pooling kernel launch_maxpool picks for these arguments.
const char *maxpool_kernel_name(int dt, int nimg, int H, int W, int C, int P,
                                int Q, int k, int stride);
hipError_t launch_maxpool(int dt, const void *x, void *y, int nimg, int H,
                          int W, int C, int P, int Q, int k, int stride,
                          int pad, hipStream_t st);
hipError_t launch_gap(int dt, const void *x, void *y, int nimg, int HW,
                      int C, hipStream_t st);

// Input assembly work item (pinned host memory): src >= 0 converts image
// src of the caller's NCHW fp32 batch into ring slot `slot` (if >= 0) and
// pass row `row` (if >= 0); src < 0 copies ring slot `slot` to row `row`.
struct StageEnt {
    int32_t src, slot, row, pad_;
};

// dt_in / dt_w / dt_out in {DT_F32, DT_F16}
hipError_t launch_fc(int dt_in, int dt_w, int dt_out, const FcArgs &a,
                     hipStream_t st);
// Whether fc_k takes its small-layer configuration (O * I <= 64 K); the
// other layers run on fc_sk, whose weights are stored in 64-row blocks.
bool fc_small(const FcArgs &a);
bool fc_small_shape(int O, int I);
// Bytes of a.part launch_fc needs for this layer and a.nimg images (0: none);
// the k-range count behind it depends on the layer's shape only.
size_t fc_part_bytes(int dt_w, const FcArgs &a);
// Name of the kernel launch_fc runs for these types and sizes.
const char *fc_kernel_name(int dt_in, int dt_w, int dt_out, const FcArgs &a);
// Global average pooling + a small fp32 FC in one kernel: a.x is the
// [nimg][HW][I] fp32 feature map; results identical to launch_gap followed
// by launch_fc.  Needs fc_small(a), I % 4 == 0, I <= GAP_FC_MAXI.
constexpr int GAP_FC_MAXI = 512;
bool gap_fc_ok(const FcArgs &a);
hipError_t launch_gap_fc(const FcArgs &a, int HW, hipStream_t st);

// Input assembly for a pass: NCHW fp32 -> NHWC (Cs <= 4 channels, zero
// padded) in dt, per the n work items of `ents` (pinned); ring and t0 hold
// [..][H][W][Cs] images.  Also copies nrows RowEnt from rows_host (pinned)
// to rows_dev when nrows > 0, and the flag bytes of `fc`.
hipError_t launch_assemble(int dt, const float *x, int C, int H, int W,
                           int Cs, const StageEnt *ents, int n, void *ring,
                           void *t0, const RowEnt *rows_host,
                           RowEnt *rows_dev, int nrows, FlagCopy fc,
                           hipStream_t st);

// Detector over a pass (Sec. II-B), when it cannot be fused into the final
// FC: for each first-execution row, flag = !(|S - ref| <= tau) with S =
// rows[r].out[col], written to rows[r].flags and flag_pass[r] (0 for
// re-executions).
hipError_t launch_verify_pass(const RowEnt *rows, int n, int col, float ref,
                              float tau, uint8_t *flag_pass, hipStream_t st);

// Detector on a strided vector: flags[i] = !(|S[i*ld] - ref| <= tau),
// *count and the ascending indices of flagged entries (each output may be
// null).
hipError_t launch_verify(const float *S, int nb, int ld, float ref, float tau,
                         uint8_t *flags, int32_t *count, int32_t *idx,
                         hipStream_t st);

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
