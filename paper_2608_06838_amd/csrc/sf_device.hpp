// sf_device.hpp -- device-side building blocks for the gfx950 (CDNA4) kernels:
// MFMA wrappers, LDS fragment loads, global->LDS tile staging with an in-register
// transpose, and wave64 scans.
//
// MFMA lane maps (measured on gfx950):
//   v_mfma_f32_16x16x32_bf16: lane l supplies A[l%16][8*(l/16)+j] and
//     B[8*(l/16)+j][l%16], j = 0..7, and receives D[4*(l/16)+r][l%16], r = 0..3.
//   v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16], B[l/16][l%16]; same D.
// Every product below is an "NT" product C[m][n] += sum_k A[m][k] * B[n][k] with
// both operands stored with the contraction index contiguous, so one fragment
// loader serves both sides.  An fp32 "k-step of 32" is eight 16x16x4 MFMAs over
// the same 8-element fragments, so bf16 and fp32 kernels share all index maths.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sf {

constexpr int C = 64;     // kernel-level chunk (tokens)
constexpr float LOG2E = 1.4426950408889634f;

// Computed bf16 MFMA operands (decayed scores, decayed keys/queries, states)
// are carried as hi + lo bf16 pairs (x = hi + lo to ~2^-17 relative), so the
// only bf16 rounding left on the dense path is that of the inputs and outputs.
#ifndef SF_SPLIT_BF16
#define SF_SPLIT_BF16 1
#endif
// per operand class (compile-time switches for accuracy/throughput studies):
// the state as an MFMA operand (S, G), the decayed per-token operands of the
// state updates, and the decayed score tiles
#ifndef SF_SPLIT_STATE
#define SF_SPLIT_STATE SF_SPLIT_BF16
#endif
#ifndef SF_SPLIT_DECAY
#define SF_SPLIT_DECAY SF_SPLIT_BF16
#endif
#ifndef SF_SPLIT_SCORES
#define SF_SPLIT_SCORES SF_SPLIT_BF16
#endif
template <typename T> constexpr bool kSplit = sizeof(T) == 2 && SF_SPLIT_BF16;
template <typename T> constexpr bool kSplitState = sizeof(T) == 2 && SF_SPLIT_STATE;
template <typename T> constexpr bool kSplitDecay = sizeof(T) == 2 && SF_SPLIT_DECAY;
template <typename T> constexpr bool kSplitScores = sizeof(T) == 2 && SF_SPLIT_SCORES;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

template <typename T> struct Frag;
template <> struct Frag<__bf16> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x8 type; };
template <typename T> using frag_t = typename Frag<T>::type;

// LDS rows are padded by 32 bytes: on gfx950 the 16-row x 16-byte fragment
// reads are conflict-free when the row pitch is 32 modulo 64 bytes (measured
// with SQ_LDS_BANK_CONFLICT over pitches 256..576 B).
template <typename T> constexpr int pad() { return 32 / (int)sizeof(T); }

// Natural tiles [token][channel] keep each 32-channel group permuted so that
// physical columns 8q..8q+7 hold logical channels {4q..4q+3, 16+4q..16+4q+3}:
// a plain 16-byte fragment read then returns the slot order of an accumulator
// pair (frag_from_acc / split_acc).  Products that contract two natural tiles
// see the same permutation on both sides and are unaffected.
__device__ __forceinline__ int nat_pos(int l) {
    const int g = l & ~31, r = l & 31;
    return g + (r < 16 ? 8 * (r >> 2) + (r & 3) : 8 * ((r - 16) >> 2) + 4 + (r & 3));
}

__device__ __forceinline__ void mma(f32x4 &c, const bf16x8 &a, const bf16x8 &b) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4 &c, const f32x8 &a, const f32x8 &b) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
}

template <typename T> __device__ __forceinline__ T cvt(float x) { return (T)x; }
template <typename T> __device__ __forceinline__ float tof(T x) { return (float)x; }

// Fragment of rows row0..row0+15, contraction columns k0..k0+31 (lane gets
// row row0 + l%16, columns k0 + 8*(l/16) .. +7).
template <typename T>
__device__ __forceinline__ frag_t<T> ldfrag(const T *base, int ld, int row0, int k0, int lane) {
    const T *p = base + (row0 + (lane & 15)) * ld + k0 + 8 * (lane >> 4);
    return *reinterpret_cast<const frag_t<T> *>(p);
}

// Transposed tiles [rows][C tokens] keep their 16-byte token blocks XOR-swizzled
// by (row >> 4): with this layout both the per-thread transposed stores and the
// 16-row fragment reads touch every LDS bank at most once per pass.
template <typename T>
__device__ __forceinline__ int tswz(int row, int t) {
    constexpr int TPB = 16 / (int)sizeof(T), NB = C / TPB;
    return (((t / TPB) ^ ((row >> 4) & (NB - 1))) * TPB) + (t % TPB);
}
// ldfrag() for a swizzled transposed tile.
template <typename T>
__device__ __forceinline__ frag_t<T> ldfragT(const T *base, int ldt, int row0, int k0, int lane) {
    const int r = row0 + (lane & 15), t = k0 + 8 * (lane >> 4);
    const T *p = base + r * ldt;
    if constexpr (sizeof(T) == 2) {
        return *reinterpret_cast<const frag_t<T> *>(p + tswz<T>(r, t));
    } else {
        f32x4 lo = *reinterpret_cast<const f32x4 *>(p + tswz<T>(r, t));
        f32x4 hi = *reinterpret_cast<const f32x4 *>(p + tswz<T>(r, t + 4));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
}

// Operand fragment built from two accumulator tiles X[m0..m0+15][n] (a0) and
// X[m0+16..m0+31][n] (a1): as an A operand it is X^T rows n, contraction over m.
template <typename T>
__device__ __forceinline__ frag_t<T> frag_from_acc(const f32x4 &a0, const f32x4 &a1) {
    frag_t<T> f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        f[j] = cvt<T>(a0[j]);
        f[j + 4] = cvt<T>(a1[j]);
    }
    return f;
}

// Fragment with every element multiplied by a per-slot factor (fp32), re-rounded.
template <typename T>
__device__ __forceinline__ frag_t<T> scale_frag(const frag_t<T> &f, const float *s) {
    frag_t<T> o;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = cvt<T>(tof<T>(f[j]) * s[j]);
    return o;
}

// Buffer addressing.  A resource (four scalar registers) covers `bytes` bytes
// from `base`; an access names it plus a 32-bit per-lane byte offset and a
// uniform (scalar) byte offset, so a tile costs one VGPR per row instead of a
// 64-bit address, and accesses past `bytes` read zero / are dropped.  The
// third word 0x00020000 selects raw (unswizzled, untyped) 32-bit addressing.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
template <typename V>
__device__ __forceinline__ V buf_ld(rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef unsigned u2 __attribute__((ext_vector_type(2)));
    typedef unsigned u4 __attribute__((ext_vector_type(4)));
    if constexpr (sizeof(V) == 16) return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
    else if constexpr (sizeof(V) == 8) return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
    else {
        static_assert(sizeof(V) == 4, "buffer load width");
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
    }
}
template <typename V>
__device__ __forceinline__ void buf_st(rsrc_t r, uint32_t voff, uint32_t soff, const V &v) {
    typedef unsigned u2 __attribute__((ext_vector_type(2)));
    typedef unsigned u4 __attribute__((ext_vector_type(4)));
    if constexpr (sizeof(V) == 16) __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), r, voff, soff, 0);
    else if constexpr (sizeof(V) == 8) __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u2, v), r, voff, soff, 0);
    else {
        static_assert(sizeof(V) == 4, "buffer store width");
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, voff, soff, 0);
    }
}
// 4 consecutive fp32 values stored as T through a buffer resource
template <typename T>
__device__ __forceinline__ void st4_buf(rsrc_t r, uint32_t voff, uint32_t soff, const f32x4 &v) {
    if constexpr (sizeof(T) == 2) buf_st(r, voff, soff, bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]});
    else buf_st(r, voff, soff, v);
}
// Bytes spanned by C rows of D elements at row stride `ld` (elements).
template <typename T, int D>
__host__ __device__ __forceinline__ uint32_t chunk_span(int64_t ld) {
    return (uint32_t)(((int64_t)(C - 1) * ld + D) * (int64_t)sizeof(T));
}

// Store 4 consecutive fp32 values as T (8 bytes for bf16, 16 for fp32).
__device__ __forceinline__ void st4(__bf16 *p, float a, float b, float c, float d) {
    bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4 *>(p) = v;
}
__device__ __forceinline__ void st4(float *p, float a, float b, float c, float d) {
    f32x4 v = {a, b, c, d};
    *reinterpret_cast<f32x4 *>(p) = v;
}
__device__ __forceinline__ f32x4 ld4f(const __bf16 *p) {
    bf16x4 v = *reinterpret_cast<const bf16x4 *>(p);
    return f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}
__device__ __forceinline__ f32x4 ld4f(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }

// 4 fp32 values rounded to T (a register-held output vector)
template <typename T>
__device__ __forceinline__ auto pack4(const f32x4 &x) {
    typedef T v4 __attribute__((ext_vector_type(4)));
    return __builtin_convertvector(x, v4);
}

// hi/lo split of 8 fp32 values: hi = T(x), lo = T(x - hi)
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void split8(const float *x, frag_t<T> &hi, frag_t<T> &lo) {
    if constexpr (sizeof(T) == 2) {
        // pairs: one packed conversion for hi, hi back to fp32 by a shift / mask of
        // the packed word, one packed conversion for lo
        typedef float f2 __attribute__((ext_vector_type(2)));
        typedef __bf16 b2 __attribute__((ext_vector_type(2)));
        typedef uint32_t u4 __attribute__((ext_vector_type(4)));
        u4 h, l;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const f2 xv = {x[2 * p], x[2 * p + 1]};
            const uint32_t u = __builtin_bit_cast(uint32_t, __builtin_convertvector(xv, b2));
            h[p] = u;
            if constexpr (SP) {
                const f2 r = {x[2 * p] - __builtin_bit_cast(float, u << 16),
                              x[2 * p + 1] - __builtin_bit_cast(float, u & 0xffff0000u)};
                l[p] = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, b2));
            }
        }
        hi = __builtin_bit_cast(frag_t<T>, h);
        if constexpr (SP) lo = __builtin_bit_cast(frag_t<T>, l);
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            hi[j] = cvt<T>(x[j]);
            lo[j] = cvt<T>(0.f);
        }
    }
}
// split fragment of two accumulator tiles (see frag_from_acc)
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void split_acc(const f32x4 &a0, const f32x4 &a1, frag_t<T> &hi, frag_t<T> &lo) {
    float x[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
    split8<T, SP>(x, hi, lo);
}
// The same fragment in plain channel order: lane row q receives channels
// 8q .. 8q+7 of the 32-channel block instead of {4q..4q+3, 16+4q..16+4q+3}.
// A 32-lane swap (rows 2,3 of the first tile with rows 0,1 of the second)
// then a 16-lane swap (odd rows of the first with even rows of the second)
// put A_{2r}, A_{2r+1} (or B_{2r-4}, B_{2r-3}) in lane row r, so such a
// fragment contracts with a tile stored in plain channel order.
__device__ __forceinline__ void acc_pair_to_plain(float (&x)[8]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        unsigned a = __builtin_bit_cast(unsigned, x[j]), b = __builtin_bit_cast(unsigned, x[4 + j]);
        const auto s32 = __builtin_amdgcn_permlane32_swap(a, b, false, false);
        const auto s16 = __builtin_amdgcn_permlane16_swap(s32[0], s32[1], false, false);
        x[j] = __builtin_bit_cast(float, (unsigned)s16[0]);
        x[4 + j] = __builtin_bit_cast(float, (unsigned)s16[1]);
    }
}
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void split_acc_plain(const f32x4 &a0, const f32x4 &a1, frag_t<T> &hi, frag_t<T> &lo) {
    float x[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
    acc_pair_to_plain(x);
    split8<T, SP>(x, hi, lo);
}
// split fragment of a T fragment scaled per slot by s[] (fp32)
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void split_scaled(const frag_t<T> &f, const float *s, frag_t<T> &hi, frag_t<T> &lo) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = tof<T>(f[j]) * s[j];
    split8<T, SP>(x, hi, lo);
}
// acc += a * b, with a given as a hi/lo pair (lo skipped when not splitting)
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void mma2(f32x4 &c, const frag_t<T> &ahi, const frag_t<T> &alo, const frag_t<T> &b) {
    mma(c, ahi, b);
    if constexpr (SP) mma(c, alo, b);
}
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void mma2b(f32x4 &c, const frag_t<T> &a, const frag_t<T> &bhi, const frag_t<T> &blo) {
    mma(c, a, bhi);
    if constexpr (SP) mma(c, a, blo);
}
// 4 consecutive fp32 values stored as a hi/lo pair of T vectors
template <typename T, bool SP = kSplit<T>>
__device__ __forceinline__ void st4_split(T *hi, T *lo, const float *v) {
    if constexpr (SP) {
        float h[4], l[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const T x = cvt<T>(v[j]);
            h[j] = tof<T>(x);
            l[j] = v[j] - h[j];
        }
        st4(hi, h[0], h[1], h[2], h[3]);
        st4(lo, l[0], l[1], l[2], l[3]);
    } else {
        st4(hi, v[0], v[1], v[2], v[3]);
    }
}

// A chunk tile of C tokens x D channels moving global -> registers -> LDS.
// Thread `tid` owns rows (tokens) row0 .. row0+RPT-1 and one 16-byte column
// block cb (E channels), so 8..16 consecutive lanes read one contiguous row.
template <typename T, int D, int NT>
struct Tile {
    static constexpr int E = 16 / (int)sizeof(T);
    static constexpr int CB = D / E;
    static constexpr int RPT = C * D / (NT * E);
    static_assert(NT % CB == 0 && RPT >= 2, "tile shape");
    typedef T vecE __attribute__((ext_vector_type(E)));
    typedef T vecR __attribute__((ext_vector_type(RPT)));
    vecE r[RPT];

    __device__ __forceinline__ int cb(int tid) const { return tid % CB; }
    __device__ __forceinline__ int row0(int tid) const { return (tid / CB) * RPT; }

    __device__ __forceinline__ void load(const T *base, int64_t row_stride, int tid) {
        const T *p = base + (int64_t)row0(tid) * row_stride + cb(tid) * E;
#pragma unroll
        for (int j = 0; j < RPT; ++j) r[j] = *reinterpret_cast<const vecE *>(p + (int64_t)j * row_stride);
    }
    // byte offsets of this thread's rows from a chunk's first token (row stride
    // in elements); one set serves every tile with that stride
    __device__ __forceinline__ static void offsets(uint32_t (&o)[RPT], int64_t row_stride, int tid) {
#pragma unroll
        for (int j = 0; j < RPT; ++j)
            o[j] = (uint32_t)(((int64_t)((tid / CB) * RPT + j) * row_stride + (tid % CB) * E) * (int64_t)sizeof(T));
    }
    __device__ __forceinline__ void load_buf(rsrc_t rs, const uint32_t (&o)[RPT], uint32_t soff) {
#pragma unroll
        for (int j = 0; j < RPT; ++j) r[j] = buf_ld<vecE>(rs, o[j], soff);
    }
    // natural layout [token][channel] (channels permuted by nat_pos), row pitch ld
    __device__ __forceinline__ void store_nat(T *lds, int ld, int tid) const {
        T *p = lds + row0(tid) * ld;
        const int ch = cb(tid) * E;
        if constexpr (E == 8) {
            typedef T half_t __attribute__((ext_vector_type(4)));
            const int p0 = nat_pos(ch), p1 = nat_pos(ch + 4);
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                *reinterpret_cast<half_t *>(p + j * ld + p0) = __builtin_shufflevector(r[j], r[j], 0, 1, 2, 3);
                *reinterpret_cast<half_t *>(p + j * ld + p1) = __builtin_shufflevector(r[j], r[j], 4, 5, 6, 7);
            }
        } else {
            const int p0 = nat_pos(ch);
#pragma unroll
            for (int j = 0; j < RPT; ++j) *reinterpret_cast<vecE *>(p + j * ld + p0) = r[j];
        }
    }
    // natural layout [token][channel] in plain channel order, rows with bit 3 set
    // XOR-swizzled by swx channels (see swz_col)
    __device__ __forceinline__ void store_swz(T *lds, int ld, int tid, int swx) const {
        const int ch = cb(tid) * E, r0 = row0(tid);
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const int row = r0 + j;
            *reinterpret_cast<vecE *>(lds + row * ld + (ch ^ (((row >> 3) & 1) * swx))) = r[j];
        }
    }
    // swizzled transposed layout [channel][token] (see tswz), token j scaled by s[j]
    __device__ __forceinline__ void store_T(T *lds, int ldt, int tid, const float *s) const {
        const int c0 = cb(tid) * E, t0 = row0(tid);
#pragma unroll
        for (int i = 0; i < E; ++i) {
            vecR vals;
#pragma unroll
            for (int j = 0; j < RPT; ++j) vals[j] = cvt<T>(tof<T>(r[j][i]) * s[j]);
            put_T(lds + (c0 + i) * ldt, c0 + i, t0, vals);
        }
    }
    // transposed, unscaled (a pure register transpose)
    __device__ __forceinline__ void store_T1(T *lds, int ldt, int tid) const {
        const int c0 = cb(tid) * E, t0 = row0(tid);
#pragma unroll
        for (int i = 0; i < E; ++i) {
            vecR vals;
#pragma unroll
            for (int j = 0; j < RPT; ++j) vals[j] = r[j][i];
            put_T(lds + (c0 + i) * ldt, c0 + i, t0, vals);
        }
    }
    // swizzled transposed layout with each scaled value kept as hi (lds) + lo (lds_lo)
    __device__ __forceinline__ void store_T2(T *lds, T *lds_lo, int ldt, int tid, const float *s) const {
        if constexpr (!kSplit<T>) {
            store_T(lds, ldt, tid, s);
        } else {
            const int c0 = cb(tid) * E, t0 = row0(tid);
#pragma unroll
            for (int i = 0; i < E; ++i) {
                vecR hi, lo;
#pragma unroll
                for (int j = 0; j < RPT; ++j) {
                    const float x = tof<T>(r[j][i]) * s[j];
                    hi[j] = cvt<T>(x);
                    lo[j] = cvt<T>(x - tof<T>(hi[j]));
                }
                put_T(lds + (c0 + i) * ldt, c0 + i, t0, hi);
                put_T(lds_lo + (c0 + i) * ldt, c0 + i, t0, lo);
            }
        }
    }
    // RPT consecutive tokens of one transposed row; split at 16-byte blocks
    __device__ __forceinline__ static void put_T(T *row, int c, int t0, const vecR &vals) {
        if constexpr (RPT * sizeof(T) <= 16) {
            *reinterpret_cast<vecR *>(row + tswz<T>(c, t0)) = vals;
        } else {
            static_assert(RPT * sizeof(T) == 32, "transposed store width");
            typedef T half_t __attribute__((ext_vector_type(RPT / 2)));
            const half_t lo = __builtin_shufflevector(vals, vals, 0, 1, 2, 3);
            const half_t hi = __builtin_shufflevector(vals, vals, 4, 5, 6, 7);
            *reinterpret_cast<half_t *>(row + tswz<T>(c, t0)) = lo;
            *reinterpret_cast<half_t *>(row + tswz<T>(c, t0 + RPT / 2)) = hi;
        }
    }
};

// ---------------------------------------------------------------------------
// Natural tiles read through transposing loads.
//
// A natural tile M[token][channel] (row pitch ld) can serve as an MFMA operand
// whose rows are channels and whose contraction runs over tokens: on gfx950,
// ds_read_b64_tr_b16 lets each group of 16 lanes exchange 4x4 blocks of 16-bit
// elements while reading.  Measured lane map: within a 16-lane group, lane i
// receives element (i % 4) of the 8-byte words addressed by lanes 4m + i/4,
// m = 0..3.  The 32-lane halves of the instruction are served together, so the
// two 16-lane groups of a half (tokens 8q.., 8(q+1)..) must hit different banks:
// rows with bit 3 set are stored with their channel index XORed by swx (128
// bytes; 64 for 128-byte rows), which made the pattern conflict-free
// (SQ_LDS_BANK_CONFLICT = 0 at a 288-byte pitch).
template <typename T, int D>
constexpr int swx() { return (D * (int)sizeof(T) >= 256 ? 128 : 64) / (int)sizeof(T); }
__device__ __forceinline__ int swz_col(int row, int col, int swx) { return col ^ (((row >> 3) & 1) * swx); }

// Per-lane element offsets into a swizzled natural tile.  Every row a lane
// touches in a fragment read has the same bit 3, and every channel of a
// fragment the same swx bit, so the swizzle reduces to +swx for channel blocks
// with that bit clear and -swx where it is set: two offsets per lane, and each
// fragment address is one of them plus a compile-time constant.
struct LaneOff {
    int lo, hi;
};
// for ldfragTR: rows k0 + 8q + (a / 4) (+4), channels c0 + 4 (a % 4) (bf16) or
// rows k0 + 8q + j, channel c0 + a (fp32), with a = lane % 16
template <typename T, int LD, int SWX>
__device__ __forceinline__ LaneOff tr_off(int lane) {
    const int q = lane >> 4, a = lane & 15, S = (q & 1) * SWX;
    const int base = sizeof(T) == 2 ? (8 * q + (a >> 2)) * LD + 4 * (a & 3) : 8 * q * LD + a;
    return {base + S, base - S};
}
// for ldfragTR with channel runs 8 apart (bf16): rows k0 + 8q + (a / 4) (+4),
// channels c0 + 8 (a % 4), so fragment row n is channel c0 + 8 (n / 4) + n % 4
template <typename T, int LD, int SWX>
__device__ __forceinline__ LaneOff tr_off8(int lane) {
    const int q = lane >> 4, a = lane & 15, S = (q & 1) * SWX;
    const int base = (8 * q + (a >> 2)) * LD + 8 * (a & 3);  // (16-bit tiles only)
    return {base + S, base - S};
}
// for ldfrag_swz: rows row0 + n, channels k0 + 8q .. +7
template <typename T, int LD, int SWX>
__device__ __forceinline__ LaneOff swz_off(int lane) {
    const int q = lane >> 4, n = lane & 15, S = ((n >> 3) & 1) * SWX;
    return {n * LD + 8 * q + S, n * LD + 8 * q - S};
}

// Lane (q = l/16, n = l%16) receives M[k0 + 8q + j][c0 + n], j = 0..7: an operand
// fragment with rows = channels c0..c0+15 and contraction = tokens k0..k0+31
// (k0 a multiple of 32, c0 of 16; o = tr_off(lane)).
template <typename T, int LD, int SWX>
__device__ __forceinline__ frag_t<T> ldfragTR(const T *M, const LaneOff &o, int k0, int c0) {
    const int e = ((c0 & SWX) ? o.hi : o.lo) + k0 * LD + c0;
    if constexpr (sizeof(T) == 2) {
        typedef short s4 __attribute__((ext_vector_type(4)));
        typedef short s8 __attribute__((ext_vector_type(8)));
        const s4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + e));
        const s4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + e + 4 * LD));
        const s8 v = __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(frag_t<T>, v);
    } else {
        frag_t<T> f = {};
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = M[e + j * LD];
        return f;
    }
}
// ldfrag() on a swizzled natural tile (rows row0.., channels k0 + 8q .. +7;
// row0 a multiple of 16, k0 of 32; o = swz_off(lane)).
template <typename T, int LD, int SWX>
__device__ __forceinline__ frag_t<T> ldfrag_swz(const T *M, const LaneOff &o, int row0, int k0) {
    return *reinterpret_cast<const frag_t<T> *>(M + ((k0 & SWX) ? o.hi : o.lo) + row0 * LD + k0);
}
// Fragment in plain channel order (channels k0 + 8q .. +7) from a tile stored
// in nat_pos order: the 8 channels sit in two 4-channel runs 8 apart.
template <typename T>
__device__ __forceinline__ frag_t<T> ldfrag_unperm(const T *M, int ld, int row0, int k0, int lane) {
    const int q = lane >> 4;
    const T *p = M + (row0 + (lane & 15)) * ld + k0 + 16 * (q & 1) + 4 * (q >> 1);
    typedef T h4 __attribute__((ext_vector_type(4)));
    const h4 lo = *reinterpret_cast<const h4 *>(p);
    const h4 hi = *reinterpret_cast<const h4 *>(p + 8);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// x summed over the four 16-lane rows of the wave (lanes l, l^16, l^32, l^48),
// returned in every lane: a 32-lane and a 16-lane swap, no LDS round trip.
__device__ __forceinline__ float sum_rows(float x) {
    const unsigned u = __builtin_bit_cast(unsigned, x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = __builtin_bit_cast(float, (unsigned)a[0]) + __builtin_bit_cast(float, (unsigned)a[1]);
    const unsigned v = __builtin_bit_cast(unsigned, y);
    const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return __builtin_bit_cast(float, (unsigned)b[0]) + __builtin_bit_cast(float, (unsigned)b[1]);
}

// Compiler scheduling fence: no instruction moves across it.  Used to keep a
// batch of LDS fragment reads ahead of independent VALU work, so that their
// latency overlaps that work instead of stalling the MFMA that consumes them.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Wait for every outstanding vector memory operation of this wave.  Loads and
// stores share one counter on gfx9-class GPUs, and once both kinds are pending
// the compiler can only wait for a load by draining everything, stores
// included.  The chunk loops therefore retire their prefetch loads here, before
// they issue the chunk's global stores, so that the next chunk's use of the
// prefetched registers does not wait for those stores.
__device__ __forceinline__ void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Inclusive prefix sum over the 64 lanes of a wave with DPP row shifts and row
// broadcasts (no LDS round trips); lanes without a source add 0.
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ float dpp_or0(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROWS, 0xf, true));
}
__device__ __forceinline__ float wave_scan_dpp(float x) {
    x += dpp_or0<0x111>(x);       // row_shr:1
    x += dpp_or0<0x112>(x);       // row_shr:2
    x += dpp_or0<0x114>(x);       // row_shr:4
    x += dpp_or0<0x118>(x);       // row_shr:8
    x += dpp_or0<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
    x += dpp_or0<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
    return x;
}
// x from lane + N of the same 16-lane row, 0 past the row's end (DPP row_shl:N)
template <int N>
__device__ __forceinline__ float dpp_row_shl(float x) { return dpp_or0<0x100 + N>(x); }
__device__ __forceinline__ float lane_value(float x, int l) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l));
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ float wave_incl_scan(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        float y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    return x;
}
// Inclusive suffix sum over the 64 lanes of a wave.
__device__ __forceinline__ float wave_incl_suffix(float x, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        float y = __shfl_down(x, o, 64);
        if (lane + o < 64) x += y;
    }
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

}  // namespace sf
