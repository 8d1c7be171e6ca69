// Device kernels of the subgraph executor and their host-side launchers.
// Every launcher enqueues on the given stream and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace byoc {

typedef uint16_t bf16_t;  // raw bfloat16 bits

enum ActCode { kActNone = 0, kActRelu = 1, kActRelu6 = 2, kActGelu = 3, kActLeaky = 4 };

// Implicit-GEMM convolution (and dense, as a 1x1 conv on 1x1 images) on
// bf16 MFMA.  Activations NHWC with Cp channels (multiple of 8); weights
// packed [rows >= Kp][Kgp] with the reduction index kk = (r*S + s)*Cp + c.
struct ConvParams {
  const bf16_t* x;
  const bf16_t* w;
  const float* bias;  // [>= Kp] (zero-padded) or nullptr
  const bf16_t* res;  // [M][ldr] or nullptr
  bf16_t* y;          // [M][ldy]
  float* partial;     // split-K: [splits][M][Kp] fp32 partial sums, else nullptr
  int N, H, W, Cp;
  int P, Q, R, S;
  int sh, sw, pt, pl;
  int M;    // N*P*Q output pixels
  int Kp;   // output channels written (multiple of 8)
  int Kg;   // R*S*Cp reduction length
  int Kgp;  // packed weight row stride (multiple of 64)
  int ldy, ldr;
  int act;
  float alpha;  // leaky ReLU slope (act == kActLeaky)
  int splits;   // split-K factor (1 = none)
  int k_tiles_per_split;
  int x_bytes;  // extent of x, w and res in bytes (buffer-load range; < 2^31)
  int w_bytes;
  int res_bytes;
  int res_post;  // 1: the residual is added after the activation, to its bf16-rounded value
  // conv_dma tile placement: > 0 splits the tile grid into (8 / xcd_py) x
  // xcd_py blocks along (pixels, channels), one per XCD, so that an XCD's L2
  // holds only its share of both operands; 0 deals tiles out linearly.
  int xcd_py;
  // Exact division by the runtime divisors of the index math, as
  // floor(n / d) = (n * mg) >> 40 with mg = ceil(2^40 / d), valid while
  // n * d < 2^40 (checked when the launch is planned).  Set by the kernel
  // launchers (the tile divisor depends on the tile shape).
  uint64_t mg_pq, mg_q, mg_cp, mg_s;
  uint64_t mg_tile;  // divisor: channel tiles per row of the tile grid (or per XCD block)
  uint64_t mg_wp, mg_hp;  // conv_halo: divisors W + 2 and H + 2 (set by its launcher)
};

inline uint64_t magic40(int d) { return ((uint64_t(1) << 40) + (uint64_t)d - 1) / (uint64_t)d; }

struct ConvTile {
  int bm, bn;       // pixels x channels per workgroup
  int mf = 16;      // MFMA shape: 16 (16x16x32) or 32 (32x32x16)
  int stages = 0;   // > 0: HBM->LDS pipeline of that many stages (conv_dma)
  int threads = 256;  // conv_dma workgroup size: 256 (4 waves) or 512 (8 waves)
  int kgroups = 1;    // conv_dma reduction groups (2: two 4-wave groups split the reduction stages)
  int halo = 0;       // 1: conv_halo kernel (stages = weight ring depth, lp / npb as planned)
  int lp = 0, npb = 0;
  int bnv = -1;       // fused bottleneck block: the kernel variant
};

// Tile configurations with a compiled kernel.
bool conv_mfma_tile_supported(int bm, int bn, int mf);
hipError_t launch_conv_mfma(const ConvParams& p, ConvTile t, hipStream_t s);
// Direct HBM->LDS pipelined variant (16x16x32 MFMA only).
bool conv_dma_tile_supported(int bm, int bn, int stages, int threads, int kgroups);
hipError_t launch_conv_dma(const ConvParams& p, int bm, int bn, int stages, int threads, int kgroups,
                           hipStream_t s);
// 3x3 stride-1 pad-1 convolution that stages each 64-channel slice of the
// input window of a tile (its output pixels' rows plus a one-pixel halo) in
// LDS once and forms all nine taps from it; weights stream per tap through
// a ring of `stages` LDS buffers.  Requires Cp % 64 == 0, P == H, Q == W.
// The reduction runs slice by slice (tap, then channel within the slice).
// conv_halo_plan checks the shape and picks the patch capacity (loads per
// thread, lp) and the number of patch buffers (npb) for a tiling; the
// launcher takes them as planned.  `stages` is the weight ring: 2 or 3
// stages of three taps (one kernel row), or 4, 6 or 8 stages of one tap.
// Tiles (bm x bn): 128 x 64 at every ring depth, 64 x 64 with 2 or 3
// stages; both sum in the same order, so they give the same bits.
bool conv_halo_plan(const ConvParams& p, int bm, int bn, int stages, int* lp, int* npb, bool i8 = false);
hipError_t launch_conv_halo(const ConvParams& p, int bm, int bn, int stages, int lp, int npb, hipStream_t s);
// Fused stem: conv (C <= 4 NCHW input channels, 64 output channels) + bias
// + activation followed by max pooling; output NHWC bf16 with 64 channels.
struct StemParams {
  const void* x;  // graph input [N][C][H][W], bf16 or f32
  int x_bf16;
  const void* w;  // packed [64][wld] bf16 (int8 codes: bytes), column r*32 + s*4 + c
  int wld;
  const void* bias;  // [64] float or nullptr (int8 codes: [64][2] {folded bias, factor bits})
  void* y;           // [N][PO][QO][64] bf16 (int8 codes)
  // int8 codes (i8 = 1): the input's 1 / scale and zero point, the conv
  // output's zero point and activation clamp in codes
  int i8;
  float inv_scale;
  int zx, zy, lo, hi;
  int N, C, H, W;
  int R, S, sh, sw, pt, pl;      // conv
  int P, Q;                      // conv output size
  int kph, kpw, sph, spw, ppt, ppl;  // pool window, stride, padding
  int PO, QO;                    // pool output size
  int act;
  float alpha;                   // leaky ReLU slope
  int grid_cap;                  // > 0: at most this many workgroups
};
bool stem_supported(int C, int K, int R, int S, int sh, int sw, int kph, int kpw, int sph, int spw);
int stem_weight_ld(int R);
int stem_weight_ld_i8(int R);  // bytes: kernel rows in pairs of 64, + 16
hipError_t launch_stem_conv_maxpool(const StemParams& p, hipStream_t s);
hipError_t launch_pack_stem_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R, int S, int wld,
                                    hipStream_t s);
// Fused bottleneck block of three conv composites and its residual:
//   m1 = act1(conv1x1(x; w1, stride S) + b1)  CIN -> F channels
//   m2 = act2(conv3x3(m1; w2, pad 1) + b2)    F -> F
//   r  = x (COUT == CIN, S == 1), or the projection conv1x1(x; wp, stride S) + bp
//   y  = act3(conv1x1(m2; w3) + b3 + r)       F -> COUT
// each intermediate rounded as the unfused composites store it; m1, m2 and
// the projection never leave the workgroup.  x NHWC [N][H][W][CIN], y
// [N][P][Q][COUT] (P, Q: the output grid of the strided 1x1); weights packed
// as for the implicit-GEMM kernels ([rows][ld], kk = (r*3 + s)*F + c for w2).
// bf16 (i8 = false): biases fp32 zero-padded to >= 256 entries (b3, bp: >=
// COUT); activations none, ReLU or ReLU6.  int8 codes (i8 = true): weights
// int8, b* the int8 conv's per-channel table {bias with the input zero
// point folded in, float32 factor bits} (>= 128 entries, b3 and bp >= COUT),
// each composite's output zero point and clamp in qz / qlo / qhi (0: m1,
// 1: m2, 2: y, 3: the projection), y = clamp(qz[2] + rescale(sum + bias,
// factor) + rescale(r - zr, mr)).  A kind (i8, F, CIN, COUT, S) has variants
// (output tile, rings); all variants of a kind sum in the same order, so
// they agree bit for bit.
struct BottleneckParams {
  const void* x;
  void* y;
  const void* w1;
  const void* w2;
  const void* w3;
  const void* wp;  // projection weights (COUT != CIN or S != 1), else unused
  const void* b1;
  const void* b2;
  const void* b3;
  const void* bp;
  int N, H, W, P, Q;
  int ld1, ld2, ld3, ldp;  // packed weight row strides (elements)
  int x_bytes, y_bytes, w1_bytes, w2_bytes, w3_bytes, wp_bytes, b1_bytes, b2_bytes, b3_bytes, bp_bytes;
  int act1, act2, act3;
  float alpha1, alpha2, alpha3;
  int qz[4], qlo[4], qhi[4];  // int8: output zero points and clamps
  int zr;                     // int8: the residual's zero point
  float mr;                   //   and its rescaling factor into y's scale
  // set by the launcher: output tiles per row band, per image and in all,
  // tiles per XCD, and the 40-bit reciprocals of the first two
  int tiles_w, tiles_hw, tiles, per_xcd;
  uint64_t mg_tw, mg_thw;
};
// Variants of a kind (0: no compiled kernel), their names, and the
// workgroups (output tiles) of variant v on an N x P x Q output.
int bottleneck_variants(bool i8, int F, int CIN, int COUT, int S);
const char* bottleneck_variant_name(bool i8, int F, int CIN, int COUT, int S, int v);
int bottleneck_tiles(bool i8, int F, int CIN, int COUT, int S, int v, int N, int P, int Q);
hipError_t launch_bottleneck(const BottleneckParams& p, bool i8, int F, int CIN, int COUT, int S, int v,
                             hipStream_t s);
// Fused MobileNetV2 inverted-residual block (bf16):
//   e = act_e(conv1x1(x; we) + be)            CIN -> F (absent: e = x, F == CIN)
//   d = act_d(depthwise3x3(e; wd, stride S, pad 1) + bd)
//   y = act_p(conv1x1(d; wp) + bp [+ x])      F -> COUT (the block input added when S == 1, CIN == COUT)
// each intermediate rounded to bf16 as the unfused composites store it; e and
// d never leave the workgroup.  x NHWC [N][H][W][CIN], y [N][P][Q][COUT];
// we / wp packed as for the implicit-GEMM kernel (row strides ldE / ldP
// elements), wd the depthwise taps [9][F] as float32 values of the bf16
// weights the depthwise kernel uses, biases fp32 zero-padded (be,
// bd >= F entries, bp >= COUT).  Channel counts are multiples of 8, CIN <= 64.
struct IrParams {
  const void* x;
  void* y;
  const void* we;
  const void* be;
  const void* wd;
  const void* bd;
  const void* wp;
  const void* bp;
  int N, H, W, P, Q, S;
  int CIN, F, COUT;
  int ldE, ldP;
  int x_bytes, y_bytes, we_bytes, be_bytes, wd_bytes, bd_bytes, wp_bytes, bp_bytes;
  int act_e, act_d, act_p;
  float alpha_e, alpha_d, alpha_p;
  int res;
  // set by the launcher: tiles per row band, per image and in all, tiles per
  // XCD, and the 40-bit reciprocals of the first two
  int tiles_w, tiles_hw, tiles, per_xcd;
  uint64_t mg_tw, mg_thw;
};
// Variants of a kind (0: no compiled kernel), their names, and the
// workgroups (output tiles) of variant v on an N x P x Q output; all
// variants of a kind give the same bits.
int ir_block_variants(int cin, int f, int cout, int s);
const char* ir_block_name(int cin, int f, int cout, int s, int v);
int ir_block_tiles(int cin, int f, int cout, int s, int v, int N, int P, int Q);
hipError_t launch_ir_block(const IrParams& p, int v, hipStream_t s);
// Plain matrix product of at most 64 rows (R = S = H = W = 1, no split):
// one workgroup per 16 output channels, the reduction split over its waves.
bool dense_rows_supported(const ConvParams& p);
hipError_t launch_dense_rows(const ConvParams& p, hipStream_t s);
// Sums split-K partials in a fixed order and applies bias, residual, act.
hipError_t launch_splitk_reduce(const ConvParams& p, hipStream_t s);

// fp32 direct convolution over NCHW with generic groups (1 or depthwise);
// dense is the 1x1 case on [M, K, 1, 1].
struct ConvF32Params {
  const float* x;
  const float* w;  // OIHW [K][C/groups][R][S]
  const float* bias;
  const float* res;  // NCHW like y, or nullptr
  float* y;
  int N, C, H, W, K, P, Q, R, S, sh, sw, pt, pl, groups, act;
  float alpha;  // leaky ReLU slope
};
hipError_t launch_conv_f32(const ConvF32Params& p, hipStream_t s);

// Depthwise conv NHWC bf16: weights packed [R*S][Cp] bf16, bias fp32 [Cp].
struct DwParams {
  const bf16_t* x;
  const bf16_t* w;
  const float* bias;
  const bf16_t* res;
  bf16_t* y;
  int N, H, W, Cp, P, Q, R, S, sh, sw, pt, pl, act;
  float alpha;  // leaky ReLU slope
};
hipError_t launch_depthwise(const DwParams& p, hipStream_t s);

struct PoolParams {
  const void* x;
  void* y;
  int N, C, H, W, Cp, P, Q, R, S, sh, sw, pt, pl;
  int ldy;  // NHWC bf16 kernels: output pixel stride in elements (0: Cp), e.g. a channel slice of a concatenation
};
hipError_t launch_maxpool_nhwc_bf16(const PoolParams& p, hipStream_t s);
hipError_t launch_avgpool_nhwc_bf16(const PoolParams& p, hipStream_t s);  // y [N][Cp]
hipError_t launch_maxpool_nchw_f32(const PoolParams& p, hipStream_t s);
// Windowed average pool NHWC bf16 (fp32 sum of the window's taps inside the
// image, divided by their count, or by R*S with count_include_pad).
hipError_t launch_avgpool_win_nhwc_bf16(const PoolParams& p, bool count_include_pad, hipStream_t s);
// Copies [pixels][C] bf16 (source pixel stride src_ld) into a channel slice
// of a concatenation (destination pixel stride dst_ld); C, src_ld, dst_ld
// multiples of 8 and 16-byte aligned bases.
hipError_t launch_copy_channels_bf16(const bf16_t* src, int src_ld, bf16_t* dst, int dst_ld, int64_t pixels, int C,
                                     hipStream_t s);
hipError_t launch_avgpool_nchw_f32(const PoolParams& p, hipStream_t s);   // y [N][C]

// y = act(a + b) over n elements (n multiple of 8 for bf16).
hipError_t launch_add_bf16(const bf16_t* a, const bf16_t* b, bf16_t* y, int64_t n, int act, float alpha,
                           hipStream_t s);
hipError_t launch_add_f32(const float* a, const float* b, float* y, int64_t n, int act, float alpha,
                          hipStream_t s);

// Boundary transforms.  src_bf16 / dst_bf16 select the external dtype.
hipError_t launch_nchw_to_nhwc(const void* x, bool src_bf16, bf16_t* y, int N, int C, int H,
                               int W, int Cp, hipStream_t s);
hipError_t launch_nhwc_to_nchw(const bf16_t* x, void* y, bool dst_bf16, int N, int C, int H,
                               int W, int Cp, hipStream_t s);
// Row-major [M, K] <-> [M, Kp] bf16 with cast.
hipError_t launch_rows_to_padded(const void* x, bool src_bf16, bf16_t* y, int M, int K, int Kp,
                                 hipStream_t s);
hipError_t launch_padded_to_rows(const bf16_t* x, void* y, bool dst_bf16, int M, int K, int Kp,
                                 hipStream_t s);
// Elementwise dtype change (fp32 graphs): f32 <-> bf16, or a plain copy.
hipError_t launch_cast(const void* x, bool src_bf16, void* y, bool dst_bf16, int64_t n,
                       hipStream_t s);

// ---- int8 (partial quantization) ------------------------------------------
// Codes are int8 with an affine (scale, zero point) per activation tensor;
// weights are symmetric per output channel.  A real rescaling factor m is
// applied in float32: rint(fl32(fl32(a) * m)), ties to even, saturated to
// +-2^20.  Activations are NHWC with Cp a multiple of 16; conv weights
// packed [rows >= Kp][Kgp] int8 with kk = (r*S + s)*Cp + c, Kgp a multiple
// of 128.
struct QConvParams {
  ConvParams g;         // geometry and operands: x, w, res, y hold int8 data; bias, partial unused
  const int32_t* qch;   // [>= Kp][2]: bias with the input zero point folded in, float32 factor bits
  const int32_t* wtap;  // [R*S][wtap_ld >= Kp] weight sums per tap (border correction), or nullptr
  int wtap_ld;
  int zx;               // input zero point (applied at the border through wtap)
  int zy, lo, hi;       // output zero point; activation clamp in output codes (within [-128, 127])
  int zr;               // residual zero point
  float mr;             // residual rescaling factor
  int leaky;            // leaky ReLU before the clamp: a negative offset from zy is scaled by slope
  float slope;
  // A following add folded in (post = 1): after the clamp, the conv's code c
  // becomes clip(pz + rescale(c - zy, pm) + rescale(res - zr, mr)), the add's
  // own arithmetic; res is then the add's other operand, not a residual.
  int post, pz;
  float pm;
};
// Tiles: 4 waves (256 threads) 128x128, 128x64, 64x64, 32x64; 8 waves (512)
// 128x128, 128x64, 64x128; 2 to 4 ring stages.  kgroups 2 or 4: that many
// 4-wave reduction groups (threads = 256 * kgroups) on 64x64 or 32x64
// tiles, 2 groups also on 128x64, as far as their rings fit the LDS.
bool conv_i8_tile_supported(int bm, int bn, int stages, int threads, int kgroups = 1);
hipError_t launch_conv_i8(const QConvParams& p, int bm, int bn, int stages, int threads, int kgroups,
                          hipStream_t s);
// The windowed 3x3 kernel on codes (conv_halo_plan(..., i8 = true) sizes it):
// 128 channels per slice; the same codes as launch_conv_i8.
hipError_t launch_conv_halo_i8(const QConvParams& q, int bm, int bn, int stages, int lp, int npb, hipStream_t s);

// Boundary Q: float NCHW (or [M, K] as N = M, C = K, H = W = 1) ->
// NHWC int8 codes clip(rint(x * inv_scale) + zp) (float32 arithmetic);
// channels past C are written as 0.
hipError_t launch_quantize_i8(const void* x, bool src_bf16, int8_t* y, int N, int C, int H, int W, int Cp,
                              float inv_scale, int zp, hipStream_t s);
// Boundary Q fused with the im2col of the conv that alone reads the input
// (an image of C <= 4 channels): y[(n*P + p)*Q + q][kk] for kk = (r*S + s)*4
// + c the code of x[n][c][p*sh - pt + r][q*sw - pl + s] (0 for c >= C), the
// zero point where that tap is outside the image, 0 for kk from 4*R*S up to
// the row length g.Cp (a multiple of 16).  Geometry in g (C, H, W, R, S,
// sh, sw, pt, pl, P, Q); R * W * 4 <= 48 KB (the input rows of one output
// row are staged in LDS).
hipError_t launch_quantize_im2col_i8(const void* x, bool src_bf16, int8_t* y, const PoolParams& g, float inv_scale,
                                     int zp, hipStream_t s);
// Boundary DQ: NHWC int8 -> float NCHW (or [M, K]) scale * (q - zp).
hipError_t launch_dequantize_i8(const int8_t* x, void* y, bool dst_bf16, int N, int C, int H, int W, int Cp,
                                float scale, int zp, hipStream_t s);
// Depthwise conv of codes, NHWC, one input channel per output channel:
// v = zy + rescale(sum over taps inside the image of (x - zx) w + bias, m)
// [+ rescale(res - zr, mr)], clamped to [lo, hi] (within [-128, 127]).
// Weights [R*S][Cp] int8; qch [>= Cp][2]: int32 bias, float32 factor bits.
struct QDwParams {
  const int8_t* x;
  const int8_t* w;
  const int32_t* qch;
  const int8_t* res;  // [N][P][Q][Cp] or nullptr
  int8_t* y;
  int N, H, W, Cp, P, Q, R, S, sh, sw, pt, pl;
  int zx, zy, lo, hi, zr;
  float mr;
  int leaky;  // leaky ReLU before the clamp (as in QConvParams)
  float slope;
};
hipError_t launch_depthwise_i8(const QDwParams& p, hipStream_t s);
// Max pooling of codes, NHWC (padding never wins).
hipError_t launch_maxpool_nhwc_i8(const PoolParams& p, hipStream_t s);
// Global average pooling of codes: y[n][c] = clip(zy + rescale(sum(x - zx), m)), y [N][Cp].
hipError_t launch_avgpool_nhwc_i8(const PoolParams& p, int zx, int zy, float m, hipStream_t s);
// y = clamp(zy + rescale(a - za, ma) + rescale(b - zb, mb), lo, hi) over n codes
// ([lo, hi] within [-128, 127]; leaky ReLU before the clamp when asked).
struct QAddParams {
  const int8_t* a;
  const int8_t* b;
  int8_t* y;
  int64_t n;
  int za, zb, zy, lo, hi;
  float ma, mb;
  int leaky;  // leaky ReLU before the clamp (as in QConvParams)
  float slope;
};
hipError_t launch_add_i8(const QAddParams& p, hipStream_t s);

// Constant packing at engine creation.
// Conv / dense weights OIHW (f32 or bf16 source) -> [rows][Kgp] bf16 with
// kk = (r*S + s)*Cp + c; zero outside the source.
hipError_t launch_pack_conv_weights(const void* src, bool src_bf16, bf16_t* dst, int K, int Cg,
                                    int R, int S, int Cp, int Kgp, int rows, hipStream_t s);
// Depthwise weights [C][1][R][S] -> [R*S][Cp] bf16.
hipError_t launch_pack_dw_weights(const void* src, bool src_bf16, bf16_t* dst, int C, int R,
                                  int S, int Cp, hipStream_t s);
// the same as float32 values of the bf16 weights
hipError_t launch_pack_dw_weights_f32(const void* src, bool src_bf16, float* dst, int C, int R, int S, int Cp,
                                      hipStream_t s);
// Vector [K] (f32 or bf16) -> fp32 [n_out], zero-padded.
hipError_t launch_pack_vector_f32(const void* src, bool src_bf16, float* dst, int K, int n_out,
                                  hipStream_t s);

}  // namespace byoc
