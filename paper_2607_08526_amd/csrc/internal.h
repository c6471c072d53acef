// Internal declarations shared by the HIP translation units of the library.
// Not part of the public interface (that is include/qlinear.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qlinear.h"

namespace qlk {

// A layer's epilogue as the kernels see it (see epilogue.h): Y[m][n] =
// act(P + bias[n]) + resid[m][n] (+ alpha * hnorm * steer[n] when
// alpha = *strength is not 0), stored as fp32 or (ybf16) bf16, and with
// ycopy also as bf16 into ycopy[m][n] (fp32 Y only).
struct Epilogue {
    const float *bias;      // [N] or nullptr
    const float *resid;     // [M][N] or nullptr
    const float *steer;     // unit direction [N] or nullptr
    const float *strength;  // device scalar alpha, read at every launch
    float hnorm;            // the layer's mean residual norm
    int act;                // QL_ACT_NONE / QL_ACT_GELU
    int ybf16;              // Y holds bf16 bit patterns
    uint16_t *ycopy;        // bf16 copy of Y [M][N] or nullptr
};

// an epilogue beyond the plain fp32 store
__host__ __device__ inline bool epi_active(const Epilogue &e)
{
    return e.bias || e.resid || e.steer || e.act || e.ybf16 || e.ycopy;
}

// Activations and packed codes of one linear layer as the kernels see it.
struct LinDesc {
    const void *X;
    const uint8_t *codes;
    const uint16_t *scales;
    float *Y;  // fp32 [M][N], or bf16 bit patterns if ep.ybf16
    Epilogue ep;
    int M, N, K;
    int tiles_m, tiles_n;
    int tile_begin;  // first logical tile of this layer in a grouped launch
    const int *xexp; // fp16 path: per-row power-of-two shift of X (see xprep.hip)
    // fp16 path, int8 / q4 weights: the power-of-two shift of each weight
    // row in each K part, wshift[part][wsld] (wsld = tiles_n * BN; set by the
    // pre-pass, xprep.hip, rows past N repeating row N - 1)
    const int *wshift;
    int wsld;
    // fp16 path, split reduction: each output tile is computed as ksplit
    // parts of psteps 64-k steps each.  cnt != nullptr (ksplit <=
    // wide_max_split()): parts store fp32 partial tiles in
    // part[tiles][ksplit][BM * BN] and count arrivals in
    // cnt[tiles_m * tiles_n] (zero before the launch); the last part to
    // arrive sums them in part order.  cnt == nullptr: parts store plain
    // partial outputs part[ksplit][M][N] and launch_split_sum adds them
    // after the launch.  ksplit == 1: no workspace.
    int ksplit, psteps;
    float *part;
    int *cnt;
    // part_out: plain partial outputs part[ksplit][M][N] (cnt == nullptr)
    // even when ksplit == 1, for a layer whose epilogue cannot take groups
    // of four outputs (N % 4 != 0 or an unaligned operand): the epilogue is
    // then applied by launch_split_sum, so the large-M kernel needs no
    // element-by-element epilogue code
    int part_out;
};

struct GroupArgs {
    LinDesc d[QL_MAX_GROUP];
    int n;
    int total_tiles;
};

// Tile shapes of the MFMA kernel (see qgemm.hip): BM rows of X by BN rows of
// W.  fp32 activations support TILE_M16..TILE_M64 only.
enum TileCfg { TILE_M16 = 0, TILE_M32 = 1, TILE_M64 = 2, TILE_M128 = 3 };

int tile_bm(TileCfg t);
int tile_bn(TileCfg t);

hipError_t launch_quantize(int fmt, const float *W, int64_t N, int64_t K, uint8_t *codes,
                           uint16_t *scales, int *status, hipStream_t stream);

// W8A8 (qgemm_w8a8.hip, quantize.hip): per-token int8 activations (one
// workgroup per row, K % 32 == 0) and their product with int8 weights.
hipError_t launch_act_quant(const void *X, bool bf16, int64_t M, int64_t K, int8_t *q,
                            uint16_t *sx, hipStream_t stream);
struct W8Args {
    const int8_t *qx;        // [M][K]
    const uint16_t *sx;      // [M] fp16 bits
    const int8_t *codes;     // [N][K]
    const uint16_t *scales;  // [N][K/32] fp16 bits
    float *Y;                // [M][N] (bf16 bit patterns if ep.ybf16)
    Epilogue ep;
    int M, N, K;
    int tiles_m, tiles_n;
};
hipError_t launch_qgemm_w8a8(const W8Args &a, hipStream_t stream);

// Fused self-attention (attention.hip), head dimension 64: Q, K, V bf16
// rows with strides (elements, multiples of 8), O fp32 or bf16.
struct AttnArgs {
    const uint16_t *q, *k, *v;
    int64_t ldq, ldk, ldv;
    void *o;
    int64_t ldo;
    int B, T, H;
    float scale_log2e;  // scale * log2(e)
    int obf16;
};
hipError_t launch_attention(const AttnArgs &a, hipStream_t stream);

// The steering injection alone, in place on h [M][N] fp32 (steer.hip).
hipError_t launch_steer(float *h, int64_t M, int64_t N, const float *dir, float hnorm,
                        const float *strength, hipStream_t stream);

hipError_t launch_qgemm(int fmt, bool xf32, TileCfg t, const GroupArgs &args,
                        hipStream_t stream);

// Large-M kernel of the fp16 path (bf16 activations): 128 x 256 tiles,
// direct-to-LDS pipeline; fmt int8, q4 or fp16 weights (QL_FMT_F16: codes
// are the fp16 weights, no scales).  Each LinDesc's X points to the fp16
// activations prepared by launch_xprep and xexp to their per-row shifts;
// K % 256 == 0 and 16-byte aligned scales.
int wide_tile_bm();
int wide_tile_bn();
int wide_max_split();
int wide_wgs_per_cu(int fmt);  // resident workgroups per CU (LDS and register budget)
hipError_t launch_qgemm_wide(int fmt, const GroupArgs &args, hipStream_t stream);

// Mid-M kernel (bf16 activations, int8 / q4 weights, exact per-block form,
// no pre-pass): 128 x 128 tiles; K % 256 == 0, K < 2^23, 16-byte aligned
// X, codes and scales; LinDesc::psteps % 4 == 0, and ksplit > 1 stores plain
// partial outputs part[ksplit][M][N] for launch_split_sum.
int mid_tile_bm();
int mid_tile_bn();
int mid_wgs_per_cu();  // resident workgroups per CU
hipError_t launch_qgemm_mid(int fmt, const GroupArgs &args, hipStream_t stream);

// Y[M][N] = sum over s < S of P[s][M][N], added in order s = 0, 1, ..., for
// n (<= QL_MAX_GROUP) split layers in one launch
struct SplitSum {
    const float *P;
    int S;
    int64_t M, N;
    float *Y;
    Epilogue ep;  // applied to the sum
};
hipError_t launch_split_sum(const SplitSum *sums, int n, hipStream_t stream);

// Slot order of an 8-k group in the q4 fp16 path: MFMA operand slot e holds
// k = Q4_SLOT[e] (the order the q4 code conversion yields; the activation
// copy is written to match).
constexpr int Q4_SLOT[8] = {0, 2, 4, 6, 1, 3, 5, 7};

// One activation tensor for the pre-pass: bf16 X [M][K] -> fp16 Xh [M][K]
// with per-row power-of-two shifts rexp[M].
struct XprepJob {
    const void *X;
    int M, K;
    uint16_t *Xh;
    int *rexp;
};
// The weight-row shifts of one int8 / q4 layer of the large-M launch:
// for K part p (blocks [p * pblocks, min((p + 1) * pblocks, nb)) of each
// row) and row n < ld, f[p * ld + n] puts qmax * (the largest scale of
// weight row min(n, N - 1) in the part) * 2^f in [2^14, 2^15) (0 for a part
// whose scales are all 0).
struct WshiftJob {
    const uint16_t *scales;  // [N][nb] fp16 bits
    int N, ld, nb, parts, pblocks, qmax;
    int *f;                  // [parts][ld]
};
struct XprepArgs {
    XprepJob j[QL_MAX_GROUP];
    int row_begin[QL_MAX_GROUP];
    int n;
    WshiftJob w[QL_MAX_GROUP];
    int wrow_begin[QL_MAX_GROUP];  // first item (part, row) of each job
    int nw;
};
// All n (<= QL_MAX_GROUP) activation jobs and nw weight-shift jobs in one
// launch, each 8-k group in Q4_SLOT order if q4_slots; also sets zero[0 ..
// nzero) to 0 (the split counters of the launch that follows on the same
// stream).
hipError_t launch_xprep(const XprepJob *jobs, int n, const WshiftJob *wjobs, int nw,
                        bool q4_slots, int *zero, int nzero, hipStream_t stream);

// Few-row kernel (bf16 activations, M <= skinny_max_m()): one layer per
// launch, workgroups of 16 weight rows with K split over their wavefronts.
int skinny_max_m();
hipError_t launch_qgemm_skinny(int fmt, const LinDesc &d, hipStream_t stream);

// Weight-streaming kernel for M <= stream_max_m() (bf16 activations): whole
// cache lines via direct-to-LDS loads; K % 256 == 0 and 16-byte aligned
// scales.
// Wavefront-reduction GEMV for M <= 4 (bf16 activations): codes and scales
// in registers, activations staged in LDS; gemv_ok() states its shape limits.
bool gemv_ok(const LinDesc &d);

int stream_max_m();
// longest reduction the streaming kernel takes: its per-lane 32-bit load
// offsets span up to 64 weight rows (64 K bytes) and 32 activation rows
int stream_max_k();
// mx: activation rows staged (8, 16, 32); rw: weight rows per workgroup;
// kw: wavefronts per workgroup (common to a group); S: the largest layer's
// K parts, psteps: the common part length in 32-blocks.  Per layer the
// LinDesc carries ksplit and psteps (ksplit > 1: LinDesc::part receives
// plain partial outputs [ksplit][M][N]).
struct StreamPlan {
    int mx, rw, kw, S, psteps;
};
// the plan of a group of n layers (one format, one M); S[i], psteps[i]
// receive each layer's parts and part length
StreamPlan stream_plan(int fmt, const LinDesc *ds, int n, int cus, int *S, int *psteps);
// n layers of one format in one launch of a few-row kernel: layer i on the
// workgroups begin[i] .. begin[i + 1] - 1 (streaming kernel: ceil(N / rw) *
// ksplit of them; GEMV: ceil(N / rows per workgroup))
struct LayerGroup {
    LinDesc d[QL_MAX_GROUP];
    int begin[QL_MAX_GROUP + 1];
    int n;
};
// The GEMV over a group of layers with one row count M (gemv_ok for each).
hipError_t launch_qgemv(int fmt, const LayerGroup &g, hipStream_t stream);
hipError_t launch_qgemm_stream(int fmt, const StreamPlan &p, const LayerGroup &g,
                               hipStream_t stream);

}  // namespace qlk
