// sf_chunk.hpp -- chunk-walk helpers shared by the scalar-gate and vector-gate
// kernels: workgroup -> (batch, head, superchunk) decode, causal tile order, exp2.
#pragma once
#include "sf_device.hpp"
#include "sf_launch.hpp"

namespace sf {

// 2^x with the hardware v_exp_f32 (results below 2^-126 flush to zero, which
// is what a decay that small means here; no input is ever > 0 except on
// masked-out causal entries, which are discarded by a select)
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// (t-tile, s-tile) pairs of the causal 64x64 score matrix, s-tile <= t-tile.
__device__ __forceinline__ void tri_tile(int i, int &tt, int &st) {
    // 0:(0,0) 1:(1,0) 2:(1,1) 3:(2,0) 4:(2,1) 5:(2,2) 6:(3,0) 7:(3,1) 8:(3,2) 9:(3,3)
    tt = (i >= 1) + (i >= 3) + (i >= 6);
    st = i - (tt * (tt + 1)) / 2;
}

// Two workgroups that share a CU progress at different rates: the issue
// arbiter favours older waves, so the workgroup dispatched first finished its
// superchunk ~25% ahead of its partner (per-workgroup timestamps), and the CU
// then ran the partner alone.  Workgroups of alternate dispatch rounds take
// turns at raised priority, in epochs of 2^12 real-time ticks (41 us at the
// 100 MHz counter), so both members of a pair progress together.
__device__ __forceinline__ unsigned pair_parity(int n_cu) { return ((int)blockIdx.x / (n_cu > 0 ? n_cu : 1)) & 1; }
__device__ __forceinline__ void pair_turn(unsigned parity) {
    if ((((unsigned)(__builtin_amdgcn_s_memrealtime() >> 12)) ^ parity) & 1) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
}

struct Decode {
    int J, bh, b, h, nch;
    int64_t tok0;
};
// item = (batch * H + head) * n_super + superchunk
__device__ __forceinline__ Decode decode(const SegArgs &a, int item) {
    Decode d;
    d.J = item % a.n_super;
    d.bh = item / a.n_super;
    d.b = d.bh / a.H;
    d.h = d.bh % a.H;
    d.tok0 = (int64_t)d.J * a.ts;
    int64_t rem = a.L - d.tok0;
    d.nch = (int)((rem < a.ts ? rem : a.ts) / C);
    return d;
}
__device__ __forceinline__ Decode decode(const SegArgs &a) { return decode(a, (int)blockIdx.x); }

}  // namespace sf
