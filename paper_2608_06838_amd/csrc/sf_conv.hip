// sf_conv.hip -- gfx950 kernels of the short convolution with a boundary tail
// (the auxiliary boundary state a segment carries next to S, Sec. 3.1):
//
//   u_t[c] = sum_{j<W} w[c][j] xh_{t-W+1+j}[c],   y_t[c] = act(u_t[c]),
//   xh_s = x_s (s >= 0), tail_in[W-1+s] (s < 0),  tail_out[i] = xh_{L-W+1+i}.
//
// Pure streaming work (W <= 4 multiply-adds per element): the roofline is HBM.
// Each thread owns 8 consecutive channels (one 16-byte row piece in bf16,
// two in fp32) of one batch and walks a block of tokens in order, keeping the
// previous W-1 inputs in registers, so every input row is read once per block
// (plus a W-1 token halo) and a wave's 64 lanes read 64 consecutive 16-byte
// pieces of a row.  Loads go out in groups of 8 tokens; outputs are written
// with non-temporal stores.
//
// Backward: du_t = dy_t * act'(u_t); dxh_s = sum_j w[j] du_{s+W-1-j} plus
// dtail_out[s-L+W-1] for the last W-1 positions; dw[c][j] = sum_{b,t} du_t
// xh_{t-W+1+j}.  A thread produces du for its tokens and the W-1 after them,
// emits dxh_s as soon as du_{s+W-1} is known, and sums its dw over its own
// tokens into a per-(batch, token block) partial; k_conv_dw_sum adds the
// partials in block order (no atomics, bitwise reproducible).
#include "sf_device.hpp"
#include "sf_launch.hpp"

namespace sf {

namespace {

constexpr int CONV_NT = 256;  // threads per workgroup
constexpr int CONV_E = 8;     // channels per thread
constexpr int CONV_G = 8;     // tokens per load group (4 and 16 measured slower)

template <typename T>
struct Row8 {
    static constexpr int NV = CONV_E * (int)sizeof(T) / 16;  // 16-byte vectors per row piece
    typedef float f4 __attribute__((ext_vector_type(4)));
    typedef unsigned u4 __attribute__((ext_vector_type(4)));
    u4 v[NV];
    __device__ __forceinline__ void load(const T *p) {
#pragma unroll
        for (int i = 0; i < NV; ++i) v[i] = reinterpret_cast<const u4 *>(p)[i];
    }
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int i = 0; i < NV; ++i) v[i] = u4{0u, 0u, 0u, 0u};
    }
    __device__ __forceinline__ void to_f32(float (&f)[CONV_E]) const {
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const unsigned w = v[0][i];
                f[2 * i] = __uint_as_float(w << 16);
                f[2 * i + 1] = __uint_as_float(w & 0xffff0000u);
            }
        } else {
#pragma unroll
            for (int i = 0; i < NV; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) f[4 * i + e] = __uint_as_float(v[i][e]);
        }
    }
};

template <typename T>
__device__ __forceinline__ void store_row8(T *p, const float (&f)[CONV_E]) {
    typedef T v8 __attribute__((ext_vector_type(8)));
    v8 o = {};
#pragma unroll
    for (int e = 0; e < CONV_E; ++e) o[e] = (T)f[e];
    // the outputs are not read again by this kernel: non-temporal stores
    // (measured 1% faster than plain stores)
    if constexpr (sizeof(T) == 2) {
        __builtin_nontemporal_store(o, reinterpret_cast<v8 *>(p));
    } else {
        typedef float f4 __attribute__((ext_vector_type(4)));
        __builtin_nontemporal_store(f4{f[0], f[1], f[2], f[3]}, reinterpret_cast<f4 *>(p));
        __builtin_nontemporal_store(f4{f[4], f[5], f[6], f[7]}, reinterpret_cast<f4 *>(p) + 1);
    }
}

__device__ __forceinline__ float sigmoid_f(float u) {
    // 1 / (1 + e^-u) through the hardware exp2; e^-u = inf for very negative u
    // gives 0, and 0 for very positive u gives 1
    return 1.f / (1.f + __builtin_amdgcn_exp2f(-u * 1.4426950408889634f));
}

template <bool SILU>
__device__ __forceinline__ float act_f(float u) {
    if constexpr (SILU) return u * sigmoid_f(u);
    else return u;
}

template <bool SILU>
__device__ __forceinline__ float dact_f(float u) {
    if constexpr (SILU) {
        const float s = sigmoid_f(u);
        return s * (1.f + u * (1.f - s));
    } else {
        return 1.f;
    }
}

// channel group of this thread, or -1 past the last one
__device__ __forceinline__ int conv_group(const ConvArgs &a) {
    const int cg = (int)blockIdx.x * CONV_NT + (int)threadIdx.x;
    return cg < a.C / CONV_E ? cg : -1;
}

// xh_s for s in [-(W-1), L): x row or tail row (zero without a tail)
template <typename T>
__device__ __forceinline__ void load_xh(const ConvArgs &a, int64_t b, int c0, int64_t s, float (&f)[CONV_E]) {
    if (s >= 0) {
        Row8<T> r;
        r.load((const T *)a.x + b * a.sx_b + s * a.sx_l + c0);
        r.to_f32(f);
    } else if (a.tail_in) {
        const float *p = a.tail_in + (b * (a.W - 1) + (a.W - 1 + s)) * (int64_t)a.C + c0;
#pragma unroll
        for (int e = 0; e < CONV_E; ++e) f[e] = p[e];
    } else {
#pragma unroll
        for (int e = 0; e < CONV_E; ++e) f[e] = 0.f;
    }
}

template <typename T, int W, bool SILU>
__global__ void __launch_bounds__(CONV_NT) k_conv_fwd(ConvArgs a) {
    const int cg = conv_group(a);
    if (cg < 0) return;
    const int c0 = cg * CONV_E;
    const int64_t b = blockIdx.z;
    const int64_t t0 = (int64_t)blockIdx.y * a.T;
    const int64_t t1 = t0 + a.T < a.L ? t0 + a.T : a.L;
    float wt[W][CONV_E];
#pragma unroll
    for (int e = 0; e < CONV_E; ++e)
#pragma unroll
        for (int j = 0; j < W; ++j) wt[j][e] = a.w[(int64_t)(c0 + e) * W + j];
    float h[W][CONV_E];  // h[j] = xh_{t-W+1+j}; h[W-1] is the current token
#pragma unroll
    for (int j = 0; j < W - 1; ++j) load_xh<T>(a, b, c0, t0 - (W - 1) + j, h[j]);
    const T *xb = (const T *)a.x + b * a.sx_b + c0;
    T *yb = (T *)a.y + b * a.sx_b + c0;
    for (int64_t tg = t0; tg < t1; tg += CONV_G) {
        Row8<T> r[CONV_G];
#pragma unroll
        for (int g = 0; g < CONV_G; ++g)
            if (tg + g < t1) r[g].load(xb + (tg + g) * a.sx_l);
#pragma unroll
        for (int g = 0; g < CONV_G; ++g) {
            if (tg + g < t1) {
                r[g].to_f32(h[W - 1]);
                float y[CONV_E];
#pragma unroll
                for (int e = 0; e < CONV_E; ++e) {
                    float u = 0.f;
#pragma unroll
                    for (int j = 0; j < W; ++j) u = fmaf(wt[j][e], h[j][e], u);
                    y[e] = act_f<SILU>(u);
                }
                store_row8<T>(yb + (tg + g) * a.sx_l, y);
#pragma unroll
                for (int j = 0; j < W - 1; ++j)
#pragma unroll
                    for (int e = 0; e < CONV_E; ++e) h[j][e] = h[j + 1][e];
            }
        }
    }
    // the block holding the last token hands on the tail xh_{L-W+1 .. L-1}
    if (W > 1 && a.tail_out && t1 == a.L) {
#pragma unroll
        for (int j = 0; j < W - 1; ++j) {
            float *p = a.tail_out + (b * (W - 1) + j) * (int64_t)a.C + c0;
#pragma unroll
            for (int e = 0; e < CONV_E; ++e) p[e] = h[j][e];
        }
    }
}

template <typename T, int W, bool SILU>
__global__ void __launch_bounds__(CONV_NT) k_conv_bwd(ConvArgs a) {
    const int cg = conv_group(a);
    if (cg < 0) return;
    const int c0 = cg * CONV_E;
    const int64_t b = blockIdx.z;
    const int64_t t0 = (int64_t)blockIdx.y * a.T;
    const int64_t t1 = t0 + a.T < a.L ? t0 + a.T : a.L;  // tokens whose dx and dw this block owns
    const int64_t tend = t1 + (W - 1);                    // du needed up to tend - 1 (zero from L on)
    float wt[W][CONV_E];
#pragma unroll
    for (int e = 0; e < CONV_E; ++e)
#pragma unroll
        for (int j = 0; j < W; ++j) wt[j][e] = a.w[(int64_t)(c0 + e) * W + j];
    float h[W][CONV_E];   // xh window of the token whose du is produced next
    float du[W][CONV_E];  // du[W-1] = du_t, du[j] = du_{t-W+1+j}
    float dw[W][CONV_E];
#pragma unroll
    for (int j = 0; j < W; ++j)
#pragma unroll
        for (int e = 0; e < CONV_E; ++e) {
            du[j][e] = 0.f;
            dw[j][e] = 0.f;
        }
#pragma unroll
    for (int j = 0; j < W - 1; ++j) load_xh<T>(a, b, c0, t0 - (W - 1) + j, h[j]);
    const T *xb = (const T *)a.x + b * a.sx_b + c0;
    const T *dyb = (const T *)a.dy + b * a.sx_b + c0;
    T *dxb = (T *)a.dx + b * a.sx_b + c0;
    const int64_t tail0 = a.L - (W - 1);  // first position that feeds tail_out
    // the first block also emits dxh_s for s < 0 (dtail_in), so it starts emitting at -(W-1)
    const int64_t s_first = t0 == 0 ? -(int64_t)(W - 1) : t0;
    for (int64_t tg = t0; tg < tend; tg += CONV_G) {
        Row8<T> rx[CONV_G], rd[CONV_G];
#pragma unroll
        for (int g = 0; g < CONV_G; ++g) {
            const int64_t t = tg + g;
            if (t < tend && t < a.L) {
                rx[g].load(xb + t * a.sx_l);
                rd[g].load(dyb + t * a.sx_l);
            }
        }
#pragma unroll
        for (int g = 0; g < CONV_G; ++g) {
            const int64_t t = tg + g;
            if (t < tend) {
#pragma unroll
                for (int j = 0; j < W - 1; ++j)
#pragma unroll
                    for (int e = 0; e < CONV_E; ++e) du[j][e] = du[j + 1][e];
                if (t < a.L) {
                    rx[g].to_f32(h[W - 1]);
                    float dy[CONV_E];
                    rd[g].to_f32(dy);
#pragma unroll
                    for (int e = 0; e < CONV_E; ++e) {
                        float u = 0.f;
#pragma unroll
                        for (int j = 0; j < W; ++j) u = fmaf(wt[j][e], h[j][e], u);
                        du[W - 1][e] = dy[e] * dact_f<SILU>(u);
                    }
                    if (t < t1) {
#pragma unroll
                        for (int j = 0; j < W; ++j)
#pragma unroll
                            for (int e = 0; e < CONV_E; ++e) dw[j][e] = fmaf(du[W - 1][e], h[j][e], dw[j][e]);
                    }
#pragma unroll
                    for (int j = 0; j < W - 1; ++j)
#pragma unroll
                        for (int e = 0; e < CONV_E; ++e) h[j][e] = h[j + 1][e];
                } else {
#pragma unroll
                    for (int e = 0; e < CONV_E; ++e) du[W - 1][e] = 0.f;
                }
                // dxh_s, s = t - W + 1, is complete: sum_j w[j] du_{s+W-1-j}
                const int64_t s = t - (W - 1);
                if (s >= s_first && s < t1) {
                    float dx[CONV_E];
#pragma unroll
                    for (int e = 0; e < CONV_E; ++e) {
                        float acc = 0.f;
#pragma unroll
                        for (int j = 0; j < W; ++j) acc = fmaf(wt[j][e], du[W - 1 - j][e], acc);
                        dx[e] = acc;
                    }
                    if (s >= tail0 && a.dtail_out) {
                        const float *p = a.dtail_out + (b * (W - 1) + (s - tail0)) * (int64_t)a.C + c0;
#pragma unroll
                        for (int e = 0; e < CONV_E; ++e) dx[e] += p[e];
                    }
                    if (s >= 0) {
                        store_row8<T>(dxb + s * a.sx_l, dx);
                    } else if (a.dtail_in) {
                        float *p = a.dtail_in + (b * (W - 1) + (W - 1 + s)) * (int64_t)a.C + c0;
#pragma unroll
                        for (int e = 0; e < CONV_E; ++e) p[e] = dx[e];
                    }
                }
            }
        }
    }
    // this block's dw partial: ws[(b * nTB + block)][c][j]
    float *pw = a.ws + ((b * a.nTB + blockIdx.y) * (int64_t)a.C + c0) * W;
#pragma unroll
    for (int e = 0; e < CONV_E; ++e)
#pragma unroll
        for (int j = 0; j < W; ++j) pw[e * W + j] = dw[j][e];
}

// dw[c][j] = sum over (batch, token block) of the partials, in that order.
// Eight partials are loaded together and then added one by one, so the loads
// overlap and the order of the additions stays fixed.
constexpr int DWS_NT = 64;
__global__ void __launch_bounds__(DWS_NT) k_conv_dw_sum(const float *ws, float *dw, int64_t n, int64_t parts) {
    const int64_t i = (int64_t)blockIdx.x * DWS_NT + threadIdx.x;
    if (i >= n) return;
    float s = 0.f;
    int64_t p = 0;
    for (; p + 8 <= parts; p += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = ws[(p + u) * n + i];
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; p < parts; ++p) s += ws[p * n + i];
    dw[i] = s;
}

// tail_out = tail_in (or zeros) when the segment is empty; dtail_in = dtail_out likewise
__global__ void __launch_bounds__(CONV_NT) k_conv_copy(const float *src, float *dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * CONV_NT + threadIdx.x;
    if (i < n) dst[i] = src ? src[i] : 0.f;
}

template <typename T, int W, bool SILU>
hipError_t conv_td(bool bwd, const ConvArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((unsigned)((a.C / CONV_E + CONV_NT - 1) / CONV_NT), (unsigned)a.nTB, (unsigned)a.B);
    if (!bwd) {
        hipExtLaunchKernelGGL((k_conv_fwd<T, W, SILU>), grid, dim3(CONV_NT), 0, s, e0, e1, 0, a);
    } else {
        hipExtLaunchKernelGGL((k_conv_bwd<T, W, SILU>), grid, dim3(CONV_NT), 0, s, e0, nullptr, 0, a);
        const int64_t n = (int64_t)a.C * W;
        hipExtLaunchKernelGGL(k_conv_dw_sum, dim3((unsigned)((n + DWS_NT - 1) / DWS_NT)), dim3(DWS_NT), 0, s,
                              nullptr, e1, 0, (const float *)a.ws, a.dw, n, (int64_t)a.B * a.nTB);
    }
    return hipGetLastError();
}

template <typename T, bool SILU>
hipError_t conv_t(bool bwd, const ConvArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    switch (a.W) {
    case 1: return conv_td<T, 1, SILU>(bwd, a, s, e0, e1);
    case 2: return conv_td<T, 2, SILU>(bwd, a, s, e0, e1);
    case 3: return conv_td<T, 3, SILU>(bwd, a, s, e0, e1);
    case 4: return conv_td<T, 4, SILU>(bwd, a, s, e0, e1);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

int conv_channels_per_thread() { return CONV_E; }

hipError_t launch_conv(bool bwd, const ConvArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (a.L == 0) {  // nothing to convolve: the tail (or its gradient) passes through
        const int64_t n = (int64_t)a.B * (a.W - 1) * a.C;
        if (bwd) {
            if (a.dtail_in && n > 0)
                hipExtLaunchKernelGGL(k_conv_copy, dim3((unsigned)((n + CONV_NT - 1) / CONV_NT)), dim3(CONV_NT), 0, s,
                                      e0, nullptr, 0, a.dtail_out, a.dtail_in, n);
            const int64_t nw = (int64_t)a.C * a.W;
            hipExtLaunchKernelGGL(k_conv_copy, dim3((unsigned)((nw + CONV_NT - 1) / CONV_NT)), dim3(CONV_NT), 0, s,
                                  (a.dtail_in && n > 0) ? nullptr : e0, e1, 0, (const float *)nullptr, a.dw, nw);
        } else if (a.tail_out && n > 0) {
            hipExtLaunchKernelGGL(k_conv_copy, dim3((unsigned)((n + CONV_NT - 1) / CONV_NT)), dim3(CONV_NT), 0, s, e0,
                                  e1, 0, a.tail_in, a.tail_out, n);
        }
        return hipGetLastError();
    }
    if (a.io == SF_BF16) return a.act ? conv_t<__bf16, true>(bwd, a, s, e0, e1) : conv_t<__bf16, false>(bwd, a, s, e0, e1);
    return a.act ? conv_t<float, true>(bwd, a, s, e0, e1) : conv_t<float, false>(bwd, a, s, e0, e1);
}

}  // namespace sf
