// sf_launch.hpp -- argument block shared by the host driver and the kernels.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "stateflow.h"

namespace sf {

// One segment (or one superchunk-parallel launch over a segment).  Token
// tensors point at the segment's first token; strides are in elements.
struct SegArgs {
    const void *q, *k, *v, *dO;
    void *o, *dq, *dk, *dv;
    const float *g;
    float *dg;
    int64_t sx_b, sx_l, sx_h;
    int64_t sg_b, sg_l, sg_h;
    int32_t B, H;
    int32_t vec;      // 1: per-key-channel gate (g, dg are [B][L][H][D])
    int32_t n_cu;     // compute units of the device
    int64_t L;        // tokens in the segment
    int32_t ts;       // superchunk length (multiple of 64)
    int32_t n_super;  // ceil(L / ts)
    const float *S_in;
    float *S_out;
    const float *dS_out;
    float *dS_in;
    float *wsS;    // [B][H][n_super][D][D]: D_J, replaced by S_J by the scan
    float *wsE;    // [B][H][n_super][D][D]: E_J, replaced by G_{J+1} (backward only)
    float *wsLg;   // [B][H][n_super] (vector gate: [..][D]): log2 of the superchunk decay
    float *wsDot;  // [B][H][n_super][D*D/256]: partials of <G_{J+1}, S_{J+1}>;
                   // vector gate: [B][H][n_super][D], the per-key-row sums
    float *wsSn;   // [B][H][D][D] or NULL: the state leaving the segment, kept
                   // beside the superchunk states when the forward keeps them
    int32_t ckpt;  // backward: 1 when wsS, wsLg and wsSn already hold the
                   // forward's superchunk states, decays and final state
};

// kind is an sf_kernel_id; io an sf_dtype.  The scan runs its backward form
// when wsE is set.  Non-null e0/e1 take the begin timestamp of the first
// kernel the kind launches and the end timestamp of its last (the timing
// rides on the dispatch packets, no marker packets are added).
hipError_t launch_kernel(int kind, int io, int D, const SegArgs &a, hipStream_t s, hipEvent_t e0 = nullptr,
                         hipEvent_t e1 = nullptr);
hipError_t launch_kernel_vg(int kind, int io, int D, const SegArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_state_copy(const float *src, float *dst, int64_t n, hipStream_t s);

// Short convolution (sf_conv.hip).  Token block T per workgroup row; nTB
// blocks per batch; ws holds B * nTB dw partials of C * W floats.
struct ConvArgs {
    const void *x;
    const float *w;
    const float *tail_in;
    void *y;
    float *tail_out;
    const void *dy;
    const float *dtail_out;
    void *dx;
    float *dw;
    float *dtail_in;
    float *ws;
    int32_t B, C, W, act, io;
    int32_t nTB;
    int64_t L, T, sx_b, sx_l;
};
int conv_channels_per_thread();

// Gated delta rule (sf_gdn.hip).  n_super superchunks of ts tokens per
// (batch, head); with n_super > 1 the workspace holds the boundary states
// wsS [B*H][n_super][D][D] and the superchunk maps wsM, wsN
// [B*H][n_prep][D][D] (all fp32; n_prep = n_super - 1 for the forward,
// n_super for the backward, which also needs M of the last superchunk).
struct GdnArgs {
    const void *q, *k, *v;
    const float *g, *beta, *S_in;
    void *o, *v_new;
    float *S_out;
    float *wsS, *wsM, *wsN;  // boundary states; superchunk maps (n_prep per head)
    float *wsSc;             // backward: the state entering every chunk [B*H][L/64][D][D]
    // backward
    const void *dO;
    const float *dS_out;
    void *dq, *dk, *dv;
    float *dg, *dbeta, *dS_in;
    float *wsE, *wsDe;  // superchunk dS offsets E_J [B*H][n_super-1], dS_end(J) [B*H][n_super]
    float *wsDc;        // dS' of every chunk [B*H][L/64][D][D]
    int32_t B, H, n_super, ts, n_prep, n_x;  // n_x: workgroups of the per-chunk gradient kernel
    int32_t scan_out;  // forward chains: maps of every superchunk, the scan writes S_out
    int64_t L, sx_b, sx_l, sx_h, sg_b, sg_l, sg_h;
};
// One kernel of the delta-rule pipeline: forward prep ([M|N] maps of the
// superchunks), scan (S_J), output walk; backward state-storing walk, dS prep
// (E_J), dS scan (dS_end(J)), dS walk, per-chunk gradients.
enum GdnPhase { GDN_PREP, GDN_SCAN, GDN_OUT, GDN_STORE, GDN_DPREP, GDN_DSCAN, GDN_DWALK, GDN_DCHUNK };
hipError_t launch_gdn_phase(int phase, const GdnArgs &a, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_conv(bool bwd, const ConvArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1);

}  // namespace sf
