// sf_abi.hip -- host side of libstateflow: argument validation, workspace
// layout, the per-segment phase sequence and the two-stream segment driver.
//
// Segment forward (paper Sec. 3.1 Fwd; phases of Sec. 2.2 Eq. 2):
//   Pre  (k_prep)  per superchunk J: D_J, Gamma_J            -- dense, MFMA
//   ST   (k_scan)  S_{J+1} = Gamma_J S_J + D_J, S_out         -- fp32 scan
//   Out  (k_walk)  walk the chunks of J from S_J, write o     -- dense, MFMA
// Segment backward (Sec. 3.1 Bwd; SR/OG/STB/PG of Sec. 3.4):
//   prep  (SR + the dO part of OG) D_J, E_J
//   scan  (ST replay + STB) S_J, G_{J+1}, dS_in
//   dq    forward walk from S_J;  dkv  reverse walk from G_{J+1}
// Chain driver (Sec. 3.1 chaining, Sec. 3.4 split-and-overlap): the scan of
// segment i runs on the aux stream while the main stream runs the prep of
// segment i+1 and the output phase of segment i-1, i.e. the schedule
// Pre(1) -> (ST(1) || Pre(2)) -> (ST(2) || Out(1)) -> Out(2) applied across
// consecutive segments; the backward mirrors it in reverse segment order.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "sf_launch.hpp"
#include "stateflow.h"

// Scratch of sf_segment_fwd_noalloc: the superchunk states and decays of one
// segment forward, for callers that cannot allocate.  One copy per GPU, held
// for the life of the process; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (the name itself is a
// host-side stand-in).  Calls that overlap on one GPU share it and race.
static __device__ __align__(256) unsigned char scratch[SF_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

sf_status fail(sf_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

sf_status hip_fail(hipError_t e, const char *what) {
    return fail(SF_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Device address of `scratch` on the current device, resolved once per device
// with that device current.
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void *g_scratch_addr[kMaxDevices];
hipError_t g_scratch_rc[kMaxDevices];

sf_status scratch_of_device(char *&out) {
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(SF_E_UNSUPPORTED, "device index %d out of range", dev);
    std::call_once(g_scratch_once[dev], [dev] {
        g_scratch_rc[dev] = hipGetSymbolAddress(&g_scratch_addr[dev], HIP_SYMBOL(scratch));
    });
    if (g_scratch_rc[dev] != hipSuccess) return hip_fail(g_scratch_rc[dev], "hipGetSymbolAddress(scratch)");
    out = (char *)g_scratch_addr[dev];
    return SF_OK;
}

// ------------------------------------------------------------- validation
struct Shape {
    int B, H, D;
    int64_t L;
    int io, gate;
    size_t esz;
    int64_t sx_b, sx_l, sx_h, sg_b, sg_l, sg_h;
};

struct Dim {
    int64_t size, stride;
};

// Strided tensor with a contiguous innermost dim of `inner` elements: the index
// map is injective iff, sorted by stride, each stride covers the previous extent.
bool non_overlapping(std::vector<Dim> dims, int64_t inner) {
    std::vector<Dim> d;
    for (auto &x : dims)
        if (x.size > 1) d.push_back(x);
    std::sort(d.begin(), d.end(), [](const Dim &a, const Dim &b) { return a.stride < b.stride; });
    int64_t extent = inner;
    for (auto &x : d) {
        if (x.stride < extent) return false;
        extent = x.stride * x.size;
    }
    return true;
}

sf_status resolve(const sf_shape *sh, Shape &r) {
    if (!sh) return fail(SF_E_NULL, "shape is NULL");
    if (sh->B < 1 || sh->H < 1 || sh->L < 0)
        return fail(SF_E_SHAPE, "need B >= 1, H >= 1, L >= 0 (got B=%d H=%d L=%lld)", sh->B, sh->H,
                    (long long)sh->L);
    if (sh->io_dtype != SF_F32 && sh->io_dtype != SF_BF16)
        return fail(SF_E_DTYPE, "unknown io_dtype %d", sh->io_dtype);
    if (sh->gate != SF_GATE_SCALAR && sh->gate != SF_GATE_VECTOR)
        return fail(SF_E_DTYPE, "unknown gate kind %d", sh->gate);
    if (sh->reserved != 0) return fail(SF_E_SHAPE, "shape.reserved must be 0");
    if (sh->Dk != sh->Dv || (sh->Dk != 64 && sh->Dk != 128))
        return fail(SF_E_UNSUPPORTED, "supported head dims: Dk == Dv in {64, 128} (got %d, %d)", sh->Dk,
                    sh->Dv);
    if (sh->chunk != 0 && sh->chunk != 64)
        return fail(SF_E_UNSUPPORTED, "chunk must be 64 (got %d)", sh->chunk);
    if (sh->L % 64 != 0) return fail(SF_E_SHAPE, "L must be a multiple of 64 (got %lld)", (long long)sh->L);
    if (sh->io_dtype == SF_F32 && sh->Dk > 64 && sh->gate == SF_GATE_VECTOR)
        return fail(SF_E_UNSUPPORTED, "fp32 I/O with the per-channel gate supports Dk <= 64 (got %d)", sh->Dk);
    r.B = sh->B;
    r.H = sh->H;
    r.D = sh->Dk;
    r.L = sh->L;
    r.io = sh->io_dtype;
    r.gate = sh->gate;
    r.esz = sh->io_dtype == SF_BF16 ? 2 : 4;
    if (sh->sx_b == 0 && sh->sx_l == 0 && sh->sx_h == 0) {
        r.sx_h = r.D;
        r.sx_l = (int64_t)r.H * r.D;
        r.sx_b = r.L * r.H * r.D;
    } else {
        r.sx_b = sh->sx_b;
        r.sx_l = sh->sx_l;
        r.sx_h = sh->sx_h;
    }
    const int64_t gin = r.gate == SF_GATE_VECTOR ? r.D : 1;
    if (sh->sg_b == 0 && sh->sg_l == 0 && sh->sg_h == 0) {
        r.sg_h = gin;
        r.sg_l = (int64_t)r.H * gin;
        r.sg_b = r.L * r.H * gin;
    } else {
        r.sg_b = sh->sg_b;
        r.sg_l = sh->sg_l;
        r.sg_h = sh->sg_h;
    }
    if (r.sx_b <= 0 || r.sx_l <= 0 || r.sx_h <= 0 || r.sg_b <= 0 || r.sg_l <= 0 || r.sg_h <= 0)
        return fail(SF_E_SHAPE, "strides must be positive");
    if (!non_overlapping({{r.B, r.sx_b}, {r.L, r.sx_l}, {r.H, r.sx_h}}, r.D))
        return fail(SF_E_SHAPE, "token-tensor strides make elements overlap");
    if (!non_overlapping({{r.B, r.sg_b}, {r.L, r.sg_l}, {r.H, r.sg_h}}, gin))
        return fail(SF_E_SHAPE, "gate strides make elements overlap");
    if ((r.sx_b * (int64_t)r.esz) % 16 || (r.sx_l * (int64_t)r.esz) % 16 || (r.sx_h * (int64_t)r.esz) % 16)
        return fail(SF_E_ALIGN, "token-tensor strides must be multiples of 16 bytes");
    // the kernels address a 64-token chunk of a tensor with 32-bit byte offsets
    if ((63 * r.sx_l + r.D) * (int64_t)r.esz >= (int64_t(1) << 31) || (63 * r.sg_l + gin) * 4 >= (int64_t(1) << 31))
        return fail(SF_E_SHAPE, "token stride too large: a 64-token chunk must span < 2 GiB");
    return SF_OK;
}

// byte extent of a tensor, as integer addresses ([lo, hi); lo = 0 for an
// absent tensor): no pointer arithmetic on absent (NULL) pointers and no
// ordering of pointers into different objects
struct Range {
    uintptr_t lo, hi;
    const char *name;
};
Range span(const void *p, int64_t bytes, const char *name) {
    const uintptr_t b = (uintptr_t)p;
    return {b, b && bytes > 0 ? b + (uintptr_t)bytes : b, name};
}
Range xrange(const Shape &r, const void *p, int64_t L, const char *name) {
    const int64_t last = (r.B - 1) * r.sx_b + (L - 1) * r.sx_l + (r.H - 1) * r.sx_h + r.D;
    return span(p, L > 0 ? last * (int64_t)r.esz : 0, name);
}
Range grange(const Shape &r, const float *p, int64_t L, const char *name) {
    const int64_t gin = r.gate == SF_GATE_VECTOR ? r.D : 1;
    const int64_t last = (r.B - 1) * r.sg_b + (L - 1) * r.sg_l + (r.H - 1) * r.sg_h + gin;
    return span(p, L > 0 ? last * 4 : 0, name);
}
Range srange(const Shape &r, const float *p, int64_t nstates, const char *name) {
    return span(p, nstates * r.B * r.H * (int64_t)r.D * r.D * 4, name);
}
Range wsrange(const void *ws, size_t bytes) { return span(ws, (int64_t)bytes, "ws"); }
bool overlap(const Range &a, const Range &b) {
    return a.lo && b.lo && a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi;
}
sf_status check_alias(const std::vector<Range> &ins, const std::vector<Range> &outs) {
    for (size_t i = 0; i < outs.size(); ++i) {
        for (auto &in : ins)
            if (overlap(outs[i], in)) return fail(SF_E_ALIAS, "output %s overlaps input %s", outs[i].name, in.name);
        for (size_t j = i + 1; j < outs.size(); ++j)
            if (overlap(outs[i], outs[j]))
                return fail(SF_E_ALIAS, "output %s overlaps output %s", outs[i].name, outs[j].name);
    }
    return SF_OK;
}
sf_status check_align(std::initializer_list<std::pair<const void *, const char *>> ps) {
    for (auto &p : ps)
        if (p.first && ((uintptr_t)p.first % 16))
            return fail(SF_E_ALIGN, "%s is not 16-byte aligned", p.second);
    return SF_OK;
}

// --------------------------------------------------------- plan / workspace
constexpr size_t ALIGN = 256;
size_t al(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

// Compute units of the current device (256 on MI355X; also the fallback when no
// device is visible, e.g. for workspace queries on a host without a GPU).
int device_cus() {
    static thread_local int cached_dev = -2, cached_cus = 256;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return 256;
    }
    if (dev != cached_dev) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
            (void)hipGetLastError();
            n = 256;
        }
        cached_dev = dev;
        cached_cus = n;
    }
    return cached_cus;
}

sf_status pick_ts(const Shape &r, int64_t L, const sf_tuning *t, int &ts) {
    if (t && t->ts != 0) {
        if (t->ts < 64 || t->ts % 64) return fail(SF_E_SHAPE, "tuning.ts must be a positive multiple of 64");
        ts = t->ts;
        return SF_OK;
    }
    // Superchunks of one head run one after another inside a workgroup.  The
    // superchunk length (a multiple of 64) minimises a cost in chunk steps,
    // fitted to measured fwd+bwd steps of five workloads (2 to 128 heads,
    // 512- to 65536-token segments):
    //   walks: m chunks per workgroup; up to one workgroup per CU they run in
    //     m steps; beyond that the CUs hold two each, in rounds of 2 * CUs,
    //     a round taking kPair * m (a second workgroup adds 1 / kPair - 1/2 of
    //     a CU's throughput); with superchunks the two prep kernels add kPrep;
    //   + kState per superchunk state of all heads (materialised, scanned and
    //     re-read: about 0.01 steps each at d = 128)
    //   + kScan per superchunk of one head (the scans' sequential steps).
    const int64_t bh = (int64_t)r.B * r.H;
    const int64_t nc = (L + 63) / 64;
    if (nc <= 1) {
        ts = (int)std::max<int64_t>(64, std::min<int64_t>(L, 1 << 30));
        return SF_OK;
    }
    const double cus = (double)device_cus(), kState = 0.01 * (double)r.D * r.D / (128.0 * 128.0);
    constexpr double kScan = 0.1, kPair = 1.6, kPrep = 1.5;
    double best = 1e300;
    int64_t best_m = nc;
    for (int64_t m = 1; m <= nc; ++m) {  // chunks per superchunk
        const int64_t ns = (nc + m - 1) / m;
        if (m > 1 && (nc + m - 2) / (m - 1) == ns) continue;  // same split as a shorter m
        const double wg = (double)(bh * ns);
        double cost = wg <= cus ? (double)m : std::ceil(wg / (2.0 * cus)) * (double)m * kPair;
        if (ns > 1) cost = cost * kPrep + kState * wg + kScan * (double)ns;
        if (cost < best - 1e-9) {
            best = cost;
            best_m = m;
        }
    }
    ts = (int)std::min<int64_t>(best_m * 64, 1 << 30);
    if (ts >= L && L > 0) ts = (int)std::min<int64_t>(L, 1 << 30);
    return SF_OK;
}

int n_super_of(int64_t L, int ts) { return L > 0 ? (int)((L + ts - 1) / ts) : 0; }

struct WsLayout {
    size_t S = 0, E = 0, Lg = 0, Dot = 0, total = 0;
};
WsLayout ws_layout(const Shape &r, int64_t L, int ts, bool bwd) {
    WsLayout w;
    const int n = n_super_of(L, ts);
    const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D;
    size_t off = 0;
    if (n > 1) {
        w.S = off;
        off += al(bh * n * SS * 4);
        if (bwd) {
            w.E = off;
            off += al(bh * n * SS * 4);
        }
        w.Lg = off;
        off += al(bh * n * (r.gate == SF_GATE_VECTOR ? r.D : 1) * 4);
    }
    if (bwd && n >= 1) {
        w.Dot = off;
        off += al(bh * n * (r.gate == SF_GATE_VECTOR ? (size_t)r.D : SS / 256) * 4);
    }
    w.total = off;
    return w;
}

// ------------------------------------------------------------- kernel timing
// The caller's timing record (sf_timing, carried by sf_tuning): a launch of a
// kernel kind whose bit is set takes the next pair of the caller's events as
// the begin and end timestamps of its own dispatch packets.  The library keeps
// nothing: the pairs, the count and the kinds live in the caller's record.
sf_status check_timing(const sf_tuning *t) {
    if (t && (t->overlap < 0 || t->overlap > 2))
        return fail(SF_E_SHAPE, "tuning.overlap must be 0, 1 or 2 (got %d)", t->overlap);
    const sf_timing *tm = t ? t->timing : nullptr;
    if (!tm) return SF_OK;
    if (tm->capacity < 0 || tm->count < 0 || tm->count > tm->capacity)
        return fail(SF_E_SHAPE, "timing: need 0 <= count <= capacity (count=%d capacity=%d)", tm->count,
                    tm->capacity);
    if (tm->capacity > 0 && (!tm->start || !tm->stop || !tm->kind))
        return fail(SF_E_NULL, "timing: start, stop and kind arrays are required");
    return SF_OK;
}
sf_timing *timing_of(const sf_tuning *t) { return t ? t->timing : nullptr; }

void take_pair(sf_timing *tm, int kind, hipEvent_t &e0, hipEvent_t &e1) {
    e0 = e1 = nullptr;
    if (!tm || kind < 0 || kind >= 32 || !((tm->mask >> kind) & 1u)) return;
    if (tm->count >= tm->capacity) {
        ++tm->dropped;
        return;
    }
    e0 = (hipEvent_t)tm->start[tm->count];
    e1 = (hipEvent_t)tm->stop[tm->count];
    tm->kind[tm->count] = kind;
    ++tm->count;
}

sf_status launch(int kind, const Shape &r, const sf::SegArgs &a, hipStream_t s, sf_timing *tm) {
    hipEvent_t e0, e1;
    take_pair(tm, kind, e0, e1);
    // the events take the dispatch timestamps of the launch itself
    hipError_t e = sf::launch_kernel(kind, r.io, r.D, a, s, e0, e1);
    return e == hipSuccess ? SF_OK : hip_fail(e, "kernel launch");
}

// ------------------------------------------------------ short convolution
struct ConvShape {
    int B, C, W, io, act;
    int64_t L, sx_b, sx_l;
    size_t esz;
};

sf_status conv_resolve(const sf_conv_shape *sh, ConvShape &r) {
    if (!sh) return fail(SF_E_NULL, "shape is NULL");
    if (sh->B < 1 || sh->C < 1 || sh->L < 0)
        return fail(SF_E_SHAPE, "need B >= 1, C >= 1, L >= 0 (got B=%d C=%d L=%lld)", sh->B, sh->C, (long long)sh->L);
    if (sh->io_dtype != SF_F32 && sh->io_dtype != SF_BF16) return fail(SF_E_DTYPE, "unknown io_dtype %d", sh->io_dtype);
    if (sh->act != SF_ACT_NONE && sh->act != SF_ACT_SILU) return fail(SF_E_DTYPE, "unknown act %d", sh->act);
    if (sh->reserved != 0) return fail(SF_E_SHAPE, "shape.reserved must be 0");
    if (sh->W < 1 || sh->W > 4) return fail(SF_E_UNSUPPORTED, "supported taps: 1 <= W <= 4 (got %d)", sh->W);
    const int ce = sf::conv_channels_per_thread();
    if (sh->C % ce) return fail(SF_E_UNSUPPORTED, "C must be a multiple of %d (got %d)", ce, sh->C);
    r.B = sh->B;
    r.C = sh->C;
    r.W = sh->W;
    r.io = sh->io_dtype;
    r.act = sh->act;
    r.L = sh->L;
    r.esz = sh->io_dtype == SF_BF16 ? 2 : 4;
    if (sh->sx_b == 0 && sh->sx_l == 0) {
        r.sx_l = r.C;
        r.sx_b = r.L * r.C;
    } else {
        r.sx_b = sh->sx_b;
        r.sx_l = sh->sx_l;
    }
    if (r.sx_b <= 0 || r.sx_l <= 0) return fail(SF_E_SHAPE, "strides must be positive");
    if (!non_overlapping({{r.B, r.sx_b}, {r.L, r.sx_l}}, r.C))
        return fail(SF_E_SHAPE, "strides make elements overlap");
    if ((r.sx_b * (int64_t)r.esz) % 16 || (r.sx_l * (int64_t)r.esz) % 16)
        return fail(SF_E_ALIGN, "strides must be multiples of 16 bytes");
    if (r.B > 65535) return fail(SF_E_UNSUPPORTED, "B must be <= 65535 (got %d)", r.B);
    return SF_OK;
}

// tokens per workgroup row: 256 in the forward; the backward grows it with L
// so that at most 256 dw partials per batch go through the workspace
int64_t conv_block(const ConvShape &r, bool bwd) {
    if (!bwd) return 256;
    const int64_t per = (r.L + 255) / 256;
    return std::max<int64_t>(256, (per + 63) / 64 * 64);
}
int64_t conv_nblocks(const ConvShape &r, bool bwd) { return (r.L + conv_block(r, bwd) - 1) / conv_block(r, bwd); }
size_t conv_ws_bytes(const ConvShape &r) {
    return r.L > 0 ? (size_t)r.B * (size_t)conv_nblocks(r, true) * (size_t)r.C * (size_t)r.W * 4 : 0;
}

Range conv_xrange(const ConvShape &r, const void *p, const char *name) {
    const int64_t last = (r.B - 1) * r.sx_b + (r.L - 1) * r.sx_l + r.C;
    return span(p, r.L > 0 ? last * (int64_t)r.esz : 0, name);
}
Range frange(const void *p, int64_t n, const char *name) { return span(p, n * 4, name); }

sf_status conv_run(int kind, bool bwd, const sf::ConvArgs &a, hipStream_t s, sf_timing *tm) {
    hipEvent_t e0, e1;
    take_pair(tm, kind, e0, e1);
    hipError_t e = sf::launch_conv(bwd, a, s, e0, e1);
    return e == hipSuccess ? SF_OK : hip_fail(e, "kernel launch");
}

// ----------------------------------------------------------- segment plans
struct Seg {
    sf::SegArgs a;
    int n;  // superchunks
    sf_timing *tm;
};

Seg make_seg(const Shape &r, int64_t L, int ts, char *ws, bool bwd, sf_timing *tm) {
    Seg s{};
    s.tm = tm;
    sf::SegArgs &a = s.a;
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    a.sx_h = r.sx_h;
    a.sg_b = r.sg_b;
    a.sg_l = r.sg_l;
    a.sg_h = r.sg_h;
    a.B = r.B;
    a.H = r.H;
    a.vec = r.gate == SF_GATE_VECTOR ? 1 : 0;
    a.n_cu = device_cus();
    a.L = L;
    a.ts = ts;
    a.n_super = n_super_of(L, ts);
    s.n = a.n_super;
    WsLayout w = ws_layout(r, L, ts, bwd);
    if (s.n > 1) {
        a.wsS = (float *)(ws + w.S);
        a.wsE = bwd ? (float *)(ws + w.E) : nullptr;
        a.wsLg = (float *)(ws + w.Lg);
    }
    if (bwd && s.n >= 1) a.wsDot = (float *)(ws + w.Dot);
    return s;
}

const char *offset_x(const Shape &r, const void *p, int64_t tok) {
    return p ? (const char *)p + tok * r.sx_l * (int64_t)r.esz : nullptr;
}
const float *offset_g(const Shape &r, const float *p, int64_t tok) { return p ? p + tok * r.sg_l : nullptr; }

// forward phases of one segment
sf_status fwd_prep(const Shape &r, const Seg &s, hipStream_t st) {
    return s.n > 1 ? launch(SF_K_FWD_PREP, r, s.a, st, s.tm) : SF_OK;
}
sf_status fwd_scan(const Shape &r, const Seg &s, hipStream_t st) {
    if (s.n > 1) return launch(SF_K_SCAN, r, s.a, st, s.tm);
    return SF_OK;
}
sf_status fwd_out(const Shape &r, const Seg &s, hipStream_t st) {
    if (s.n == 0) {
        hipError_t e = sf::launch_state_copy(s.a.S_in, s.a.S_out, (int64_t)r.B * r.H * r.D * r.D, st);
        return e == hipSuccess ? SF_OK : hip_fail(e, "state copy");
    }
    sf::SegArgs a = s.a;
    if (s.n > 1) a.S_out = nullptr;  // the scan wrote S_out
    return launch(SF_K_FWD_OUT, r, a, st, s.tm);
}
// backward phases
sf_status bwd_prep(const Shape &r, const Seg &s, hipStream_t st) {
    return s.n > 1 ? launch(SF_K_BWD_PREP, r, s.a, st, s.tm) : SF_OK;
}
sf_status bwd_scan(const Shape &r, const Seg &s, hipStream_t st) {
    return s.n > 1 ? launch(SF_K_SCAN, r, s.a, st, s.tm) : SF_OK;
}
sf_status bwd_grad(const Shape &r, const Seg &s, hipStream_t st) {
    if (s.n == 0) {
        hipError_t e = sf::launch_state_copy(s.a.dS_out, s.a.dS_in, (int64_t)r.B * r.H * r.D * r.D, st);
        return e == hipSuccess ? SF_OK : hip_fail(e, "state copy");
    }
    sf_status rc = launch(SF_K_BWD_DQ, r, s.a, st, s.tm);
    if (rc != SF_OK) return rc;
    return launch(SF_K_BWD_DKV, r, s.a, st, s.tm);
}

// ------------------------------------------------------------ stream events
struct EventPool {
    int dev = -1;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};  // dependency, join, scan done (x2)
};
thread_local EventPool g_events;

sf_status events(hipEvent_t &e0, hipEvent_t &e1, hipEvent_t *scan_done = nullptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (g_events.dev != dev) {
        for (auto &x : g_events.ev) {
            x = nullptr;
            e = hipEventCreateWithFlags(&x, hipEventDisableTiming);
            if (e != hipSuccess) return hip_fail(e, "hipEventCreateWithFlags");
        }
        g_events.dev = dev;
    }
    e0 = g_events.ev[0];
    e1 = g_events.ev[1];
    if (scan_done) {
        scan_done[0] = g_events.ev[2];
        scan_done[1] = g_events.ev[3];
    }
    return SF_OK;
}
// the main stream waits for one recorded point of the aux stream
sf_status record(hipEvent_t ev, hipStream_t s) {
    const hipError_t e = hipEventRecord(ev, s);
    return e == hipSuccess ? SF_OK : hip_fail(e, "event record");
}
sf_status wait(hipStream_t s, hipEvent_t ev) {
    const hipError_t e = hipStreamWaitEvent(s, ev, 0);
    return e == hipSuccess ? SF_OK : hip_fail(e, "stream wait");
}
sf_status dep(hipStream_t from, hipStream_t to, hipEvent_t ev) {
    if (from == to) return SF_OK;
    hipError_t e = hipEventRecord(ev, from);
    if (e == hipSuccess) e = hipStreamWaitEvent(to, ev, 0);
    return e == hipSuccess ? SF_OK : hip_fail(e, "stream dependency");
}

#define TRY(x)                          \
    do {                                \
        sf_status _rc = (x);            \
        if (_rc != SF_OK) return _rc;   \
    } while (0)

sf_status check_segments(const Shape &r, int32_t n_seg, const int64_t *seg_len) {
    if (n_seg < 1) return fail(SF_E_SHAPE, "n_seg must be >= 1");
    if (!seg_len) return fail(SF_E_NULL, "seg_len is NULL");
    int64_t sum = 0;
    for (int i = 0; i < n_seg; ++i) {
        if (seg_len[i] <= 0 || seg_len[i] % 64)
            return fail(SF_E_SHAPE, "seg_len[%d] = %lld must be a positive multiple of 64", i,
                        (long long)seg_len[i]);
        sum += seg_len[i];
    }
    if (sum != r.L) return fail(SF_E_SHAPE, "segment lengths sum to %lld, shape.L is %lld", (long long)sum,
                                (long long)r.L);
    return SF_OK;
}

// Kept superchunk states of one segment with more than one superchunk: the
// kernels' wsS (S_J after the forward scan), wsLg and wsSn regions.
struct CkptLayout {
    size_t S = 0, Lg = 0, Sn = 0, total = 0;
};
CkptLayout ckpt_layout(const Shape &r, int64_t L, int ts) {
    CkptLayout c;
    const int n = n_super_of(L, ts);
    if (n <= 1) return c;
    const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D;
    c.Lg = al(bh * n * SS * 4);
    c.Sn = c.Lg + al(bh * n * (r.gate == SF_GATE_VECTOR ? r.D : 1) * 4);
    c.total = c.Sn + al(bh * SS * 4);
    return c;
}
sf_status chain_ckpt(const Shape &r, int32_t n_seg, const int64_t *seg_len, const sf_tuning *t, size_t &bytes) {
    bytes = 0;
    for (int i = 0; i < n_seg; ++i) {
        int ts;
        TRY(pick_ts(r, seg_len[i], t, ts));
        bytes += ckpt_layout(r, seg_len[i], ts).total;
    }
    return SF_OK;
}
// point a segment's superchunk-state regions into the kept-state buffer
void use_ckpt(const Shape &r, Seg &s, char *base, bool bwd) {
    const CkptLayout c = ckpt_layout(r, s.a.L, s.a.ts);
    if (c.total == 0) return;
    s.a.wsS = (float *)(base + c.S);
    s.a.wsLg = (float *)(base + c.Lg);
    s.a.wsSn = (float *)(base + c.Sn);
    s.a.ckpt = bwd ? 1 : 0;
}

size_t chain_ws(const Shape &r, int32_t n_seg, const int64_t *seg_len, const sf_tuning *t) {
    size_t slot = 0;
    for (int i = 0; i < n_seg; ++i) {
        int ts;
        if (pick_ts(r, seg_len[i], t, ts) != SF_OK) return 0;
        slot = std::max(slot, std::max(ws_layout(r, seg_len[i], ts, true).total,
                                       ws_layout(r, seg_len[i], ts, false).total));
    }
    const size_t gbnd = al((size_t)r.B * r.H * r.D * r.D * 4);
    return 2 * al(slot) + 2 * gbnd;
}

// argument checks shared by the two segment-forward entry points; resolves the
// shape, the superchunk length and the workspace the phases need
sf_status segment_fwd_check(const sf_shape *shape, const void *q, const void *k, const void *v, const float *g,
                            const float *S_in, void *o, float *S_out, const sf_tuning *tuning, Shape &r, int &ts,
                            size_t &need) {
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    if (!S_out || (r.L > 0 && (!q || !k || !v || !g || !o)))
        return fail(SF_E_NULL, "q, k, v, g, o and S_out are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {o, "o"}, {S_in, "S_in"}, {S_out, "S_out"}}));
    TRY(pick_ts(r, r.L, tuning, ts));
    need = ws_layout(r, r.L, ts, false).total;
    return SF_OK;
}

sf_status segment_fwd_run(const Shape &r, int ts, const void *q, const void *k, const void *v, const float *g,
                          const float *S_in, void *o, float *S_out, char *ws, const sf_tuning *tuning,
                          hipStream_t st) {
    Seg s = make_seg(r, r.L, ts, ws, false, timing_of(tuning));
    s.a.q = q;
    s.a.k = k;
    s.a.v = v;
    s.a.g = g;
    s.a.o = o;
    s.a.S_in = S_in;
    s.a.S_out = S_out;
    TRY(fwd_prep(r, s, st));
    TRY(fwd_scan(r, s, st));
    TRY(fwd_out(r, s, st));
    return SF_OK;
}

// ------------------------------------------------- exact partition rounding
// The boundary c_i(alpha) = (1 - alpha) i T / N + alpha c_i^hyb, with
// A(c_i^hyb) = (i / N) A(T) and A(c) = w_tok c + w_soft c^2 / 2, is compared
// with a half-way point y = (2m + 1) R / 2 exactly, the fp64 inputs taken at
// their exact values.  With K = (2m + 1) R N, J = 2 i T, U = K - J and
// Z = U + alpha J (so y = K / 2N and c_i(alpha) >= y iff c_i^hyb >= Z / 2N alpha),
// multiplying A(Z / 2N alpha) <= (i / N) A(T) by 8 N^2 alpha^2 gives
//     c_i(alpha) >= y  iff  alpha = 0 and U <= 0,  or  Z <= 0,  or  F <= 0,
//     F = 4 N U (alpha w_tok) + U^2 w_soft + 2 U J (alpha w_soft) + 4 i T^2 (i - N) (alpha^2 w_soft).
// Every term is an integer times a product of doubles, i.e. an integer times a
// power of two; their sum is formed exactly in a fixed-size big integer.
constexpr int64_t kPartMaxT = int64_t(1) << 40;
constexpr int32_t kPartMaxN = 1 << 20;

struct BigInt {  // sign and magnitude, little-endian 64-bit limbs
    static constexpr int W = 112;  // 7168 bits: every term below, shifted by any exponent gap of three doubles
    bool neg = false;
    uint64_t w[W] = {};
    bool zero() const {
        for (uint64_t x : w)
            if (x) return false;
        return true;
    }
};
void big_mul_small(BigInt &a, uint64_t m) {
    unsigned __int128 carry = 0;
    for (int i = 0; i < BigInt::W; ++i) {
        const unsigned __int128 t = (unsigned __int128)a.w[i] * m + carry;
        a.w[i] = (uint64_t)t;
        carry = t >> 64;
    }
}
void big_shl(BigInt &a, int k) {
    const int q = k / 64, r = k % 64;
    for (int i = BigInt::W - 1; i >= 0; --i) {
        uint64_t v = i - q >= 0 ? a.w[i - q] << r : 0;
        if (r && i - q - 1 >= 0) v |= a.w[i - q - 1] >> (64 - r);
        a.w[i] = v;
    }
}
int big_cmp_mag(const BigInt &a, const BigInt &b) {
    for (int i = BigInt::W - 1; i >= 0; --i)
        if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
    return 0;
}
void big_add(BigInt &acc, const BigInt &t) {  // acc += t (signed)
    if (acc.neg == t.neg) {
        unsigned __int128 carry = 0;
        for (int i = 0; i < BigInt::W; ++i) {
            const unsigned __int128 s = (unsigned __int128)acc.w[i] + t.w[i] + carry;
            acc.w[i] = (uint64_t)s;
            carry = s >> 64;
        }
        return;
    }
    const bool acc_bigger = big_cmp_mag(acc, t) >= 0;
    const BigInt &hi = acc_bigger ? acc : t, &lo = acc_bigger ? t : acc;
    BigInt d;
    d.neg = hi.neg;
    uint64_t borrow = 0;
    for (int i = 0; i < BigInt::W; ++i) {
        const uint64_t a = hi.w[i], b = lo.w[i];
        d.w[i] = a - b - borrow;
        borrow = (a < b || (a == b && borrow)) ? 1 : 0;
    }
    acc = d;
}
// x = mant * 2^ex with mant a non-negative integer below 2^53 (x finite, >= 0)
void split_double(double x, uint64_t &mant, int &ex) {
    int e = 0;
    const double f = std::frexp(x, &e);  // x = f 2^e, 0.5 <= f < 1 (or 0)
    mant = (uint64_t)std::ldexp(f, 53);
    ex = e - 53;
}
struct Term {
    __int128 coef;   // integer factor
    int nd;          // number of doubles multiplied in
    uint64_t m[3];   // their mantissas
    int ex;          // sum of their exponents
};
// sign (-1, 0, 1) of sum_k coef_k * prod mantissas * 2^ex_k, exactly
int exact_sign(const Term *t, int n) {
    int emin = 0;
    bool any = false;
    for (int k = 0; k < n; ++k) {
        bool nz = t[k].coef != 0;
        for (int j = 0; j < t[k].nd; ++j) nz = nz && t[k].m[j] != 0;
        if (nz && (!any || t[k].ex < emin)) emin = t[k].ex;
        any = any || nz;
    }
    if (!any) return 0;
    BigInt acc;
    for (int k = 0; k < n; ++k) {
        bool nz = t[k].coef != 0;
        for (int j = 0; j < t[k].nd; ++j) nz = nz && t[k].m[j] != 0;
        if (!nz) continue;
        BigInt b;
        const unsigned __int128 mag = t[k].coef < 0 ? (unsigned __int128)(-t[k].coef) : (unsigned __int128)t[k].coef;
        b.w[0] = (uint64_t)mag;
        b.w[1] = (uint64_t)(mag >> 64);
        b.neg = t[k].coef < 0;
        for (int j = 0; j < t[k].nd; ++j) big_mul_small(b, t[k].m[j]);
        big_shl(b, t[k].ex - emin);
        big_add(acc, b);
    }
    if (acc.zero()) return 0;
    return acc.neg ? -1 : 1;
}
// exactly: is c_i(alpha) >= (odd * R) / 2 ?
bool part_at_least(int64_t T, int32_t N, int32_t i, double alpha, double w_tok, double w_soft, int32_t R,
                   int64_t odd) {
    const __int128 K = (__int128)odd * R * N, J = (__int128)2 * i * T, U = K - J;
    if (alpha == 0.0) return U <= 0;
    uint64_t ma, mp, ms;
    int ea, ep, es;
    split_double(alpha, ma, ea);
    split_double(w_tok, mp, ep);
    split_double(w_soft, ms, es);
    const Term z[2] = {{U, 0, {0, 0, 0}, 0}, {J, 1, {ma, 0, 0}, ea}};  // Z = U + alpha J
    if (exact_sign(z, 2) <= 0) return true;
    const __int128 T2 = (__int128)T * T;
    const Term f[4] = {{4 * (__int128)N * U, 2, {ma, mp, 0}, ea + ep},
                       {U * U, 1, {ms, 0, 0}, es},
                       {2 * U * J, 2, {ma, ms, 0}, ea + es},
                       {4 * (__int128)i * T2 * (i - N), 3, {ma, ma, ms}, 2 * ea + es}};
    return exact_sign(f, 4) <= 0;
}

}  // namespace

// ===================================================================== ABI
extern "C" {

int sf_abi_version(void) { return SF_ABI_VERSION; }

const char *sf_status_str(int s) {
    switch (s) {
    case SF_OK: return "SF_OK";
    case SF_E_NULL: return "SF_E_NULL";
    case SF_E_SHAPE: return "SF_E_SHAPE";
    case SF_E_DTYPE: return "SF_E_DTYPE";
    case SF_E_ALIGN: return "SF_E_ALIGN";
    case SF_E_ALIAS: return "SF_E_ALIAS";
    case SF_E_WORKSPACE: return "SF_E_WORKSPACE";
    case SF_E_UNSUPPORTED: return "SF_E_UNSUPPORTED";
    case SF_E_HIP: return "SF_E_HIP";
    default: return "SF_E_UNKNOWN";
    }
}

const char *sf_last_error(void) { return g_err.c_str(); }

size_t sf_fwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning) {
    Shape r;
    int ts;
    if (resolve(shape, r) != SF_OK || pick_ts(r, r.L, tuning, ts) != SF_OK) return 0;
    return ws_layout(r, r.L, ts, false).total;
}

size_t sf_bwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning) {
    Shape r;
    int ts;
    if (resolve(shape, r) != SF_OK || pick_ts(r, r.L, tuning, ts) != SF_OK) return 0;
    return ws_layout(r, r.L, ts, true).total;
}

sf_status sf_segment_fwd(const sf_shape *shape, const void *q, const void *k, const void *v,
                         const float *g, const float *S_in, void *o, float *S_out, void *ws,
                         size_t ws_bytes, const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    Shape r;
    int ts;
    size_t need;
    TRY(segment_fwd_check(shape, q, k, v, g, S_in, o, S_out, tuning, r, ts, need));
    TRY(check_align({{ws, "ws"}}));
    if (need > 0 && !ws) return fail(SF_E_NULL, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, need);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"),
                     grange(r, g, r.L, "g"), srange(r, S_in, 1, "S_in")},
                    {xrange(r, o, r.L, "o"), srange(r, S_out, 1, "S_out"), wsrange(ws, need)}));
    return segment_fwd_run(r, ts, q, k, v, g, S_in, o, S_out, (char *)ws, tuning, (hipStream_t)stream);
}

sf_status sf_segment_fwd_noalloc(const sf_shape *shape, const void *q, const void *k, const void *v,
                                 const float *g, const float *S_in, void *o, float *S_out,
                                 const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    Shape r;
    int ts;
    size_t need;
    TRY(segment_fwd_check(shape, q, k, v, g, S_in, o, S_out, tuning, r, ts, need));
    if (need > SF_NOALLOC_SCRATCH_BYTES)
        return fail(SF_E_WORKSPACE,
                    "this shape needs %zu bytes of scratch; the allocation-free call holds %zu "
                    "(use sf_segment_fwd with a workspace, or a larger tuning.ts)",
                    need, (size_t)SF_NOALLOC_SCRATCH_BYTES);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"),
                     grange(r, g, r.L, "g"), srange(r, S_in, 1, "S_in")},
                    {xrange(r, o, r.L, "o"), srange(r, S_out, 1, "S_out")}));
    char *ws = nullptr;
    if (need > 0) TRY(scratch_of_device(ws));
    return segment_fwd_run(r, ts, q, k, v, g, S_in, o, S_out, ws, tuning, (hipStream_t)stream);
}

sf_status sf_segment_bwd(const sf_shape *shape, const void *q, const void *k, const void *v,
                         const float *g, const float *S_in, const void *dO, const float *dS_out,
                         void *dq, void *dk, void *dv, float *dg, float *dS_in, void *ws, size_t ws_bytes,
                         const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    if (!dS_in || (r.L > 0 && (!q || !k || !v || !g || !dO || !dq || !dk || !dv || !dg)))
        return fail(SF_E_NULL, "q, k, v, g, dO, dq, dk, dv, dg and dS_in are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {dO, "dO"}, {dq, "dq"}, {dk, "dk"}, {dv, "dv"},
                     {S_in, "S_in"}, {dS_out, "dS_out"}, {dS_in, "dS_in"}, {ws, "ws"}}));
    int ts;
    TRY(pick_ts(r, r.L, tuning, ts));
    const size_t need = ws_layout(r, r.L, ts, true).total;
    if (need > 0 && !ws) return fail(SF_E_NULL, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, need);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"),
                     grange(r, g, r.L, "g"), srange(r, S_in, 1, "S_in"), xrange(r, dO, r.L, "dO"),
                     srange(r, dS_out, 1, "dS_out")},
                    {xrange(r, dq, r.L, "dq"), xrange(r, dk, r.L, "dk"), xrange(r, dv, r.L, "dv"),
                     grange(r, dg, r.L, "dg"), srange(r, dS_in, 1, "dS_in"), wsrange(ws, need)}));
    Seg s = make_seg(r, r.L, ts, (char *)ws, true, timing_of(tuning));
    s.a.q = q;
    s.a.k = k;
    s.a.v = v;
    s.a.g = g;
    s.a.dO = dO;
    s.a.dq = dq;
    s.a.dk = dk;
    s.a.dv = dv;
    s.a.dg = dg;
    s.a.S_in = S_in;
    s.a.dS_out = dS_out;
    s.a.dS_in = dS_in;
    hipStream_t st = (hipStream_t)stream;
    TRY(bwd_prep(r, s, st));
    TRY(bwd_scan(r, s, st));
    TRY(bwd_grad(r, s, st));
    return SF_OK;
}

size_t sf_chain_workspace_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                                const sf_tuning *tuning) {
    Shape r;
    if (resolve(shape, r) != SF_OK || check_segments(r, n_seg, seg_len) != SF_OK) return 0;
    return chain_ws(r, n_seg, seg_len, tuning);
}

size_t sf_chain_ckpt_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                           const sf_tuning *tuning) {
    g_err.clear();
    Shape r;
    size_t bytes = 0;
    if (resolve(shape, r) != SF_OK || check_segments(r, n_seg, seg_len) != SF_OK ||
        chain_ckpt(r, n_seg, seg_len, tuning, bytes) != SF_OK)
        return 0;
    return bytes;
}

sf_status sf_chain_fwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                       const void *k, const void *v, const float *g, void *o, float *S_bnd, void *ckpt,
                       size_t ckpt_bytes, void *ws, size_t ws_bytes, const sf_tuning *tuning, sf_stream main_s,
                       sf_stream aux_s) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    TRY(check_segments(r, n_seg, seg_len));
    if (!q || !k || !v || !g || !o || !S_bnd || !ws)
        return fail(SF_E_NULL, "q, k, v, g, o, S_bnd and ws are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {o, "o"}, {S_bnd, "S_bnd"}, {ckpt, "ckpt"}, {ws, "ws"}}));
    const size_t need = chain_ws(r, n_seg, seg_len, tuning);
    if (need == 0) return fail(SF_E_SHAPE, "cannot size the chain workspace");
    if (ws_bytes < need) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, need);
    size_t kneed = 0;
    TRY(chain_ckpt(r, n_seg, seg_len, tuning, kneed));
    if (ckpt && ckpt_bytes < kneed) return fail(SF_E_WORKSPACE, "ckpt %zu < required %zu", ckpt_bytes, kneed);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"),
                     grange(r, g, r.L, "g")},
                    {xrange(r, o, r.L, "o"), srange(r, S_bnd, n_seg + 1, "S_bnd"),
                     span(ckpt, (int64_t)kneed, "ckpt"), wsrange(ws, need)}));
    const size_t slot = (need - 2 * al((size_t)r.B * r.H * r.D * r.D * 4)) / 2;
    const int64_t SSB = (int64_t)r.B * r.H * r.D * r.D;
    hipStream_t mn = (hipStream_t)main_s;
    hipStream_t ax = (aux_s && (!tuning || tuning->overlap != 0)) ? (hipStream_t)aux_s : mn;
    const bool prep_aux = ax != mn && tuning && tuning->overlap == 2;
    hipEvent_t e0 = nullptr, e1 = nullptr, sd[2] = {nullptr, nullptr};
    if (ax != mn) TRY(events(e0, e1, sd));
    if (ax != mn) TRY(dep(mn, ax, e0));  // aux sees everything queued on main so far

    std::vector<Seg> segs(n_seg);
    int64_t tok = 0;
    size_t kofs = 0;
    for (int i = 0; i < n_seg; ++i) {
        int ts;
        TRY(pick_ts(r, seg_len[i], tuning, ts));
        Seg &s = segs[i];
        s = make_seg(r, seg_len[i], ts, (char *)ws + (i % 2) * slot, false, timing_of(tuning));
        if (ckpt) {
            use_ckpt(r, s, (char *)ckpt + kofs, false);
            kofs += ckpt_layout(r, seg_len[i], ts).total;
        }
        s.a.q = offset_x(r, q, tok);
        s.a.k = offset_x(r, k, tok);
        s.a.v = offset_x(r, v, tok);
        s.a.g = offset_g(r, g, tok);
        s.a.o = (void *)offset_x(r, o, tok);
        s.a.S_in = S_bnd + i * SSB;
        s.a.S_out = S_bnd + (i + 1) * SSB;
        tok += seg_len[i];
    }
    // Schedule (Sec. 3.4): Pre(i) -> [ST(i) on aux || Out(i-1) on main] -> Pre(i+1) ...
    // Out(i-1) waits only for ST(i-1) (its own recorded point on aux), so ST(i)
    // overlaps it.  S_bnd[i] is produced by ST(i-1) on aux (multi-superchunk
    // segments; waited for before Out(i-1), hence before a single-superchunk
    // Out(i)) or by the walk of segment i-1 on main (single-superchunk).  Two
    // workspace slots suffice: Pre(i+1) overwrites slot (i+1)%2 on main after
    // Out(i-1) has read it.
    int pending = -1;
    for (int i = 0; i < n_seg; ++i) {
        Seg &s = segs[i];
        if (s.n > 1) {
            if (prep_aux) {
                TRY(dep(mn, ax, e0));  // slot i%2 free (Out(i-2) done) and any main-side S_bnd[i] producer
                TRY(fwd_prep(r, s, ax));
            } else {
                TRY(fwd_prep(r, s, mn));
                TRY(dep(mn, ax, e0));  // prep(i) done (and any main-side S_bnd[i] producer)
            }
            TRY(fwd_scan(r, s, ax));
            if (ax != mn) TRY(record(sd[i % 2], ax));
        }
        if (pending >= 0) {
            if (ax != mn) TRY(wait(mn, sd[pending % 2]));
            TRY(fwd_out(r, segs[pending], mn));
            pending = -1;
        }
        if (s.n > 1) pending = i;
        else TRY(fwd_out(r, s, mn));
    }
    if (pending >= 0) {
        if (ax != mn) TRY(wait(mn, sd[pending % 2]));
        TRY(fwd_out(r, segs[pending], mn));
    }
    if (ax != mn) TRY(dep(ax, mn, e1));
    return SF_OK;
}

sf_status sf_chain_bwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                       const void *k, const void *v, const float *g, const float *S_bnd, const void *ckpt,
                       size_t ckpt_bytes, const void *dO, const float *dS_final, void *dq, void *dk, void *dv,
                       float *dg, float *dS_init, void *ws, size_t ws_bytes, const sf_tuning *tuning,
                       sf_stream main_s, sf_stream aux_s) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    TRY(check_segments(r, n_seg, seg_len));
    if (!q || !k || !v || !g || !S_bnd || !dO || !dq || !dk || !dv || !dg || !dS_init || !ws)
        return fail(SF_E_NULL, "q, k, v, g, S_bnd, dO, dq, dk, dv, dg, dS_init and ws are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {dO, "dO"}, {dq, "dq"}, {dk, "dk"}, {dv, "dv"},
                     {S_bnd, "S_bnd"}, {ckpt, "ckpt"}, {dS_final, "dS_final"}, {dS_init, "dS_init"},
                     {ws, "ws"}}));
    const size_t need = chain_ws(r, n_seg, seg_len, tuning);
    if (need == 0) return fail(SF_E_SHAPE, "cannot size the chain workspace");
    if (ws_bytes < need) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, need);
    size_t kneed = 0;
    TRY(chain_ckpt(r, n_seg, seg_len, tuning, kneed));
    if (ckpt && ckpt_bytes < kneed) return fail(SF_E_WORKSPACE, "ckpt %zu < required %zu", ckpt_bytes, kneed);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"),
                     grange(r, g, r.L, "g"), srange(r, S_bnd, n_seg, "S_bnd"), span(ckpt, (int64_t)kneed, "ckpt"),
                     xrange(r, dO, r.L, "dO"), srange(r, dS_final, 1, "dS_final")},
                    {xrange(r, dq, r.L, "dq"), xrange(r, dk, r.L, "dk"), xrange(r, dv, r.L, "dv"),
                     grange(r, dg, r.L, "dg"), srange(r, dS_init, 1, "dS_init"), wsrange(ws, need)}));
    const size_t gb = al((size_t)r.B * r.H * r.D * r.D * 4);
    const size_t slot = (need - 2 * gb) / 2;
    float *gbnd[2] = {(float *)((char *)ws + 2 * slot), (float *)((char *)ws + 2 * slot + gb)};
    const int64_t SSB = (int64_t)r.B * r.H * r.D * r.D;
    hipStream_t mn = (hipStream_t)main_s;
    hipStream_t ax = (aux_s && (!tuning || tuning->overlap != 0)) ? (hipStream_t)aux_s : mn;
    const bool prep_aux = ax != mn && tuning && tuning->overlap == 2;
    hipEvent_t e0 = nullptr, e1 = nullptr, sd[2] = {nullptr, nullptr};
    if (ax != mn) TRY(events(e0, e1, sd));
    if (ax != mn) TRY(dep(mn, ax, e0));

    std::vector<Seg> segs(n_seg);
    int64_t tok = 0;
    size_t kofs = 0;
    for (int i = 0; i < n_seg; ++i) {
        int ts;
        TRY(pick_ts(r, seg_len[i], tuning, ts));
        Seg &s = segs[i];
        s = make_seg(r, seg_len[i], ts, (char *)ws + (i % 2) * slot, true, timing_of(tuning));
        if (ckpt) {
            use_ckpt(r, s, (char *)ckpt + kofs, true);
            kofs += ckpt_layout(r, seg_len[i], ts).total;
        }
        s.a.q = offset_x(r, q, tok);
        s.a.k = offset_x(r, k, tok);
        s.a.v = offset_x(r, v, tok);
        s.a.g = offset_g(r, g, tok);
        s.a.dO = offset_x(r, dO, tok);
        s.a.dq = (void *)offset_x(r, dq, tok);
        s.a.dk = (void *)offset_x(r, dk, tok);
        s.a.dv = (void *)offset_x(r, dv, tok);
        s.a.dg = (float *)offset_g(r, dg, tok);
        s.a.S_in = S_bnd + i * SSB;
        s.a.dS_out = i == n_seg - 1 ? dS_final : gbnd[(i + 1) % 2];
        s.a.dS_in = i == 0 ? dS_init : gbnd[i % 2];
        tok += seg_len[i];
    }
    // Mirror of the forward schedule: the gradient kernels of segment i+1 wait
    // only for STB(i+1) and overlap STB(i).  For a multi-superchunk segment the
    // gradient kernels read G_J from their own slot, never dS_out, so STB(i)
    // writing dS_in(i) meanwhile is safe; a single-superchunk segment's
    // kernels read dS_out, produced by STB(i+1) (waited for just before) or by
    // the kernels of segment i+1 on main.
    int pending = -1;
    for (int i = n_seg - 1; i >= 0; --i) {
        Seg &s = segs[i];
        if (s.n > 1) {
            if (prep_aux) {
                TRY(dep(mn, ax, e0));  // slot i%2 free (the gradients of i+2 done) and any main-side dS producer
                TRY(bwd_prep(r, s, ax));
            } else {
                TRY(bwd_prep(r, s, mn));
                TRY(dep(mn, ax, e0));
            }
            TRY(bwd_scan(r, s, ax));
            if (ax != mn) TRY(record(sd[i % 2], ax));
        }
        if (pending >= 0) {
            if (ax != mn) TRY(wait(mn, sd[pending % 2]));
            TRY(bwd_grad(r, segs[pending], mn));
            pending = -1;
        }
        if (s.n > 1) pending = i;
        else TRY(bwd_grad(r, s, mn));
    }
    if (pending >= 0) {
        if (ax != mn) TRY(wait(mn, sd[pending % 2]));
        TRY(bwd_grad(r, segs[pending], mn));
    }
    if (ax != mn) TRY(dep(ax, mn, e1));
    return SF_OK;
}

size_t sf_conv_bwd_workspace_bytes(const sf_conv_shape *shape) {
    ConvShape r;
    if (conv_resolve(shape, r) != SF_OK) return 0;
    return conv_ws_bytes(r);
}

sf_status sf_conv_fwd(const sf_conv_shape *shape, const void *x, const float *w, const float *tail_in, void *y,
                      float *tail_out, const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    ConvShape r;
    TRY(conv_resolve(shape, r));
    TRY(check_timing(tuning));
    const bool tail = r.W > 1;
    if (!w || (r.L > 0 && (!x || !y))) return fail(SF_E_NULL, "x, w and y are required");
    TRY(check_align({{x, "x"}, {y, "y"}}));
    if (((uintptr_t)w | (uintptr_t)(tail ? tail_in : nullptr) | (uintptr_t)(tail ? tail_out : nullptr)) % 4)
        return fail(SF_E_ALIGN, "w and the tails must be 4-byte aligned");
    const int64_t nt = (int64_t)r.B * (r.W - 1) * r.C;
    TRY(check_alias({conv_xrange(r, x, "x"), frange(w, (int64_t)r.C * r.W, "w"),
                     frange(tail ? tail_in : nullptr, nt, "tail_in")},
                    {conv_xrange(r, y, "y"), frange(tail ? tail_out : nullptr, nt, "tail_out")}));
    if (r.L == 0 && (!tail || !tail_out)) return SF_OK;  // nothing to write
    sf::ConvArgs a{};
    a.x = x;
    a.w = w;
    a.tail_in = tail ? tail_in : nullptr;
    a.y = y;
    a.tail_out = tail ? tail_out : nullptr;
    a.B = r.B;
    a.C = r.C;
    a.W = r.W;
    a.act = r.act;
    a.io = r.io;
    a.L = r.L;
    a.T = conv_block(r, false);
    a.nTB = (int32_t)conv_nblocks(r, false);
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    if (a.nTB > 65535) return fail(SF_E_UNSUPPORTED, "L too large for one call (%lld tokens)", (long long)r.L);
    return conv_run(SF_K_CONV_FWD, false, a, (hipStream_t)stream, timing_of(tuning));
}

sf_status sf_conv_bwd(const sf_conv_shape *shape, const void *x, const float *w, const float *tail_in, const void *dy,
                      const float *dtail_out, void *dx, float *dw, float *dtail_in, void *ws, size_t ws_bytes,
                      const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    ConvShape r;
    TRY(conv_resolve(shape, r));
    TRY(check_timing(tuning));
    const bool tail = r.W > 1;
    if (!w || !dw || (r.L > 0 && (!x || !dy || !dx))) return fail(SF_E_NULL, "x, w, dy, dx and dw are required");
    const size_t need = conv_ws_bytes(r);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(SF_E_WORKSPACE, "workspace of %zu bytes needed (got %zu)", need, ws ? ws_bytes : (size_t)0);
    TRY(check_align({{x, "x"}, {dy, "dy"}, {dx, "dx"}}));
    if (((uintptr_t)w | (uintptr_t)dw | (uintptr_t)ws | (uintptr_t)(tail ? tail_in : nullptr) |
         (uintptr_t)(tail ? dtail_out : nullptr) | (uintptr_t)(tail ? dtail_in : nullptr)) % 4)
        return fail(SF_E_ALIGN, "w, dw, the workspace and the tails must be 4-byte aligned");
    const int64_t nt = (int64_t)r.B * (r.W - 1) * r.C, nw = (int64_t)r.C * r.W;
    TRY(check_alias({conv_xrange(r, x, "x"), frange(w, nw, "w"), frange(tail ? tail_in : nullptr, nt, "tail_in"),
                     conv_xrange(r, dy, "dy"), frange(tail ? dtail_out : nullptr, nt, "dtail_out")},
                    {conv_xrange(r, dx, "dx"), frange(dw, nw, "dw"), frange(tail ? dtail_in : nullptr, nt, "dtail_in"),
                     wsrange(ws, need)}));
    sf::ConvArgs a{};
    a.x = x;
    a.w = w;
    a.tail_in = tail ? tail_in : nullptr;
    a.dy = dy;
    a.dtail_out = tail ? dtail_out : nullptr;
    a.dx = dx;
    a.dw = dw;
    a.dtail_in = tail ? dtail_in : nullptr;
    a.ws = (float *)ws;
    a.B = r.B;
    a.C = r.C;
    a.W = r.W;
    a.act = r.act;
    a.io = r.io;
    a.L = r.L;
    a.T = conv_block(r, true);
    a.nTB = (int32_t)conv_nblocks(r, true);
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    return conv_run(SF_K_CONV_BWD, true, a, (hipStream_t)stream, timing_of(tuning));
}

}  // extern "C"

namespace {

// Gated delta rule: superchunk length.  One walk workgroup fills a CU (its
// LDS), so `slots` = CUs; the prep walk ([M | N], twice the columns) costs
// about kPrep chunk steps of the output walk per chunk and one scan step about
// kScan.  Choose chunks per superchunk m minimising
//   rounds(walk) * m + kPrep * rounds(prep) * m + kScan * (superchunks - 1).
sf_status gdn_pick_ts(const Shape &r, const sf_tuning *t, int &ts) {
    if (t && t->ts != 0) {
        if (t->ts < 64 || t->ts % 64) return fail(SF_E_SHAPE, "tuning.ts must be a positive multiple of 64");
        ts = t->ts;
        return SF_OK;
    }
    const int64_t bh = (int64_t)r.B * r.H, nc = r.L / 64;
    if (nc <= 1) {
        ts = 64;
        return SF_OK;
    }
    const double slots = device_cus(), kPrep = 1.3, kScan = 0.15;
    double best = 1e300;
    int64_t best_m = nc;
    for (int64_t m = 1; m <= nc; ++m) {
        const int64_t ns = (nc + m - 1) / m;
        if (m > 1 && (nc + m - 2) / (m - 1) == ns) continue;
        const double walk = std::ceil((double)(bh * ns) / slots) * (double)m;
        const double prep = ns > 1 ? kPrep * std::ceil((double)(bh * (ns - 1)) / slots) * (double)m : 0.0;
        const double cost = walk + prep + kScan * (double)(ns - 1);
        if (cost < best - 1e-9) {
            best = cost;
            best_m = m;
        }
    }
    ts = (int)std::min<int64_t>(best_m * 64, 1 << 30);
    return SF_OK;
}

size_t gdn_ws_bytes(const Shape &r, int ts) {
    const int n = n_super_of(r.L, ts);
    if (n <= 1) return 0;
    const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D * 4;
    return al(bh * n * SS) + 2 * al(bh * (n - 1) * SS);
}

// Backward workspace: the forward's boundary states and maps (M, N for every
// superchunk), E_J and dS_end(J), and the state and the state gradient of
// every chunk.  n_x: workgroups of the per-chunk gradient kernel (one per CU).
struct GdnBwdWs {
    size_t S = 0, M = 0, N = 0, E = 0, De = 0, Sc = 0, Dc = 0, total = 0;
    int n_x = 0;
};
// for n superchunks and nc chunks per (batch, head)
GdnBwdWs gdn_bwd_ws_n(const Shape &r, int n, size_t nc) {
    GdnBwdWs w;
    const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D * 4;
    size_t off = 0;
    auto take = [&](size_t &at, size_t bytes) {
        at = off;
        off += al(bytes);
    };
    if (n > 1) {
        take(w.S, bh * n * SS);
        take(w.M, bh * n * SS);
        take(w.N, bh * n * SS);
        take(w.E, bh * (n - 1) * SS);
        take(w.De, bh * n * SS);
    }
    take(w.Sc, std::max<size_t>(bh * nc * SS, 1));
    take(w.Dc, std::max<size_t>(bh * nc * SS, 1));
    w.n_x = (int)std::max<size_t>(1, std::min<size_t>(bh * nc, (size_t)device_cus()));
    w.total = off;
    return w;
}
GdnBwdWs gdn_bwd_ws(const Shape &r, int ts) { return gdn_bwd_ws_n(r, std::max(1, n_super_of(r.L, ts)), (size_t)(r.L / 64)); }

// Forward workspace: S_J for every superchunk, then M, N for n_prep of them.
struct GdnFwdWs {
    size_t S = 0, M = 0, N = 0, total = 0;
};
GdnFwdWs gdn_fwd_ws_n(const Shape &r, int n, int n_prep) {
    GdnFwdWs w;
    if (n <= 1) return w;
    const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D * 4;
    w.M = al(bh * n * SS);
    w.N = w.M + al(bh * n_prep * SS);
    w.total = w.N + al(bh * n_prep * SS);
    return w;
}

// GdnArgs of tokens [tok, tok + L) of the shape's tensors (pointers of the
// whole-sequence tensors; NULL stays NULL).
sf::GdnArgs gdn_seg_args(const Shape &r, int64_t tok, int64_t L, int ts, const void *q, const void *k,
                         const void *v, const float *g, const float *beta) {
    sf::GdnArgs a{};
    a.q = offset_x(r, q, tok);
    a.k = offset_x(r, k, tok);
    a.v = offset_x(r, v, tok);
    a.g = offset_g(r, g, tok);
    a.beta = offset_g(r, beta, tok);
    a.B = r.B;
    a.H = r.H;
    a.L = L;
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    a.sx_h = r.sx_h;
    a.sg_b = r.sg_b;
    a.sg_l = r.sg_l;
    a.sg_h = r.sg_h;
    a.ts = ts;
    a.n_super = std::max(1, n_super_of(L, ts));
    return a;
}

// superchunk length and count of every segment, and the largest of each
struct GdnPlan {
    std::vector<int> ts, n;
    int n_max = 1;
    int64_t nc_max = 0;
};
sf_status gdn_plan(const Shape &r, int32_t n_seg, const int64_t *seg_len, const sf_tuning *t, GdnPlan &p) {
    p.ts.resize(n_seg);
    p.n.resize(n_seg);
    for (int i = 0; i < n_seg; ++i) {
        Shape rs = r;
        rs.L = seg_len[i];
        TRY(gdn_pick_ts(rs, t, p.ts[i]));
        p.n[i] = std::max(1, n_super_of(seg_len[i], p.ts[i]));
        p.n_max = std::max(p.n_max, p.n[i]);
        p.nc_max = std::max<int64_t>(p.nc_max, seg_len[i] / 64);
    }
    return SF_OK;
}
// chain workspace: two forward sets (maps of every superchunk) or one backward
// set and two boundary-gradient slots, whichever is larger
struct GdnChainWs {
    size_t fwd_set = 0, bwd = 0, dslot = 0, total = 0;
};
GdnChainWs gdn_chain_ws(const Shape &r, const GdnPlan &p) {
    GdnChainWs w;
    w.fwd_set = al(std::max<size_t>(gdn_fwd_ws_n(r, p.n_max, p.n_max).total, 1));
    w.bwd = al(gdn_bwd_ws_n(r, p.n_max, (size_t)p.nc_max).total);
    w.dslot = al((size_t)r.B * r.H * r.D * r.D * 4);
    w.total = std::max(2 * w.fwd_set, w.bwd + 2 * w.dslot);
    return w;
}

// kept states of a chain: per segment of n > 1 superchunks, S_J then M_J
size_t gdn_ckpt_seg(const Shape &r, int n) {
    return n > 1 ? 2 * al((size_t)r.B * r.H * n * (size_t)r.D * r.D * 4) : 0;
}
size_t gdn_ckpt_total(const Shape &r, const GdnPlan &p) {
    size_t t = 0;
    for (int n : p.n) t += gdn_ckpt_seg(r, n);
    return t;
}

sf_status gdn_shape_ok(const Shape &r) {
    if (r.io != SF_BF16) return fail(SF_E_UNSUPPORTED, "the gated delta rule needs bf16 I/O");
    if (r.gate != SF_GATE_SCALAR) return fail(SF_E_UNSUPPORTED, "the gated delta rule takes a scalar gate");
    return SF_OK;
}

// one kernel of the delta-rule pipeline; its timing kind is SF_K_GDN_PREP + phase
sf_status gdn_launch(int phase, const sf::GdnArgs &a, int D, hipStream_t s, sf_timing *tm) {
    if (phase == sf::GDN_DCHUNK && a.L < 64) return SF_OK;  // no chunk: nothing to launch
    hipEvent_t e0, e1;
    take_pair(tm, SF_K_GDN_PREP + phase, e0, e1);
    const hipError_t e = sf::launch_gdn_phase(phase, a, D, s, e0, e1);
    return e == hipSuccess ? SF_OK : hip_fail(e, "kernel launch");
}


// the phases of one delta-rule segment call, in order, on one stream
sf_status gdn_run_fwd(const sf::GdnArgs &a, int D, hipStream_t s, sf_timing *tm) {
    if (a.n_super > 1) {
        TRY(gdn_launch(sf::GDN_PREP, a, D, s, tm));
        TRY(gdn_launch(sf::GDN_SCAN, a, D, s, tm));
    }
    return gdn_launch(sf::GDN_OUT, a, D, s, tm);
}
sf_status gdn_run_bwd(const sf::GdnArgs &a, int D, hipStream_t s, sf_timing *tm) {
    if (a.n_super > 1) {
        TRY(gdn_launch(sf::GDN_PREP, a, D, s, tm));
        TRY(gdn_launch(sf::GDN_SCAN, a, D, s, tm));
        TRY(gdn_launch(sf::GDN_DPREP, a, D, s, tm));
        TRY(gdn_launch(sf::GDN_DSCAN, a, D, s, tm));
    }
    TRY(gdn_launch(sf::GDN_STORE, a, D, s, tm));
    TRY(gdn_launch(sf::GDN_DWALK, a, D, s, tm));
    return gdn_launch(sf::GDN_DCHUNK, a, D, s, tm);
}

}  // namespace

extern "C" {

size_t sf_gdn_fwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning) {
    Shape r;
    int ts;
    if (resolve(shape, r) != SF_OK || gdn_pick_ts(r, tuning, ts) != SF_OK) return 0;
    return gdn_ws_bytes(r, ts);
}

sf_status sf_gdn_fwd(const sf_shape *shape, const void *q, const void *k, const void *v, const float *g,
                     const float *beta, const float *S_in, void *o, float *S_out, void *v_new, void *ws,
                     size_t ws_bytes, const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    if (r.io != SF_BF16) return fail(SF_E_UNSUPPORTED, "the gated delta rule needs bf16 I/O");
    if (r.gate != SF_GATE_SCALAR) return fail(SF_E_UNSUPPORTED, "the gated delta rule takes a scalar gate");
    if (!S_out || (r.L > 0 && (!q || !k || !v || !g || !beta || !o)))
        return fail(SF_E_NULL, "q, k, v, g, beta, o and S_out are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {o, "o"}, {S_in, "S_in"}, {S_out, "S_out"}, {v_new, "v_new"},
                     {ws, "ws"}}));
    if (((uintptr_t)g | (uintptr_t)beta) % 4) return fail(SF_E_ALIGN, "g and beta must be 4-byte aligned");
    int ts;
    TRY(gdn_pick_ts(r, tuning, ts));
    const size_t need = gdn_ws_bytes(r, ts);
    if (need > 0 && !ws) return fail(SF_E_NULL, "workspace of %zu bytes required", need);
    if (ws_bytes < need) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, need);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"), grange(r, g, r.L, "g"),
                     grange(r, beta, r.L, "beta"), srange(r, S_in, 1, "S_in")},
                    {xrange(r, o, r.L, "o"), srange(r, S_out, 1, "S_out"), xrange(r, v_new, r.L, "v_new"),
                     wsrange(ws, need)}));
    sf::GdnArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.g = g;
    a.beta = beta;
    a.S_in = S_in;
    a.o = o;
    a.v_new = v_new;
    a.S_out = S_out;
    a.B = r.B;
    a.H = r.H;
    a.L = r.L;
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    a.sx_h = r.sx_h;
    a.sg_b = r.sg_b;
    a.sg_l = r.sg_l;
    a.sg_h = r.sg_h;
    a.ts = ts;
    a.n_super = std::max(1, n_super_of(r.L, ts));
    a.n_prep = a.n_super - 1;
    if (a.n_super > 1) {
        const size_t bh = (size_t)r.B * r.H, SS = (size_t)r.D * r.D * 4;
        a.wsS = (float *)ws;
        a.wsM = (float *)((char *)ws + al(bh * a.n_super * SS));
        a.wsN = (float *)((char *)a.wsM + al(bh * (a.n_super - 1) * SS));
    }
    return gdn_run_fwd(a, r.D, (hipStream_t)stream, timing_of(tuning));
}

size_t sf_gdn_bwd_workspace_bytes(const sf_shape *shape, const sf_tuning *tuning) {
    Shape r;
    int ts;
    if (resolve(shape, r) != SF_OK || gdn_pick_ts(r, tuning, ts) != SF_OK) return 0;
    return gdn_bwd_ws(r, ts).total;
}

sf_status sf_gdn_bwd(const sf_shape *shape, const void *q, const void *k, const void *v, const float *g,
                     const float *beta, const float *S_in, const void *dO, const float *dS_out, void *dq, void *dk,
                     void *dv, float *dg, float *dbeta, float *dS_in, void *ws, size_t ws_bytes,
                     const sf_tuning *tuning, sf_stream stream) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    if (r.io != SF_BF16) return fail(SF_E_UNSUPPORTED, "the gated delta rule needs bf16 I/O");
    if (r.gate != SF_GATE_SCALAR) return fail(SF_E_UNSUPPORTED, "the gated delta rule takes a scalar gate");
    if (!dS_in || (r.L > 0 && (!q || !k || !v || !g || !beta || !dO || !dq || !dk || !dv || !dg || !dbeta)))
        return fail(SF_E_NULL, "q, k, v, g, beta, dO, dq, dk, dv, dg, dbeta and dS_in are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {dO, "dO"}, {dq, "dq"}, {dk, "dk"}, {dv, "dv"}, {S_in, "S_in"},
                     {dS_out, "dS_out"}, {dS_in, "dS_in"}, {ws, "ws"}}));
    if (((uintptr_t)g | (uintptr_t)beta | (uintptr_t)dg | (uintptr_t)dbeta) % 4)
        return fail(SF_E_ALIGN, "g, beta, dg and dbeta must be 4-byte aligned");
    int ts;
    TRY(gdn_pick_ts(r, tuning, ts));
    const GdnBwdWs L = gdn_bwd_ws(r, ts);
    if (!ws) return fail(SF_E_NULL, "workspace of %zu bytes required", L.total);
    if (ws_bytes < L.total) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, L.total);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"), grange(r, g, r.L, "g"),
                     grange(r, beta, r.L, "beta"), srange(r, S_in, 1, "S_in"), xrange(r, dO, r.L, "dO"),
                     srange(r, dS_out, 1, "dS_out")},
                    {xrange(r, dq, r.L, "dq"), xrange(r, dk, r.L, "dk"), xrange(r, dv, r.L, "dv"),
                     grange(r, dg, r.L, "dg"), grange(r, dbeta, r.L, "dbeta"), srange(r, dS_in, 1, "dS_in"),
                     wsrange(ws, L.total)}));
    sf::GdnArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.g = g;
    a.beta = beta;
    a.S_in = S_in;
    a.dO = dO;
    a.dS_out = dS_out;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.dg = dg;
    a.dbeta = dbeta;
    a.dS_in = dS_in;
    a.B = r.B;
    a.H = r.H;
    a.L = r.L;
    a.sx_b = r.sx_b;
    a.sx_l = r.sx_l;
    a.sx_h = r.sx_h;
    a.sg_b = r.sg_b;
    a.sg_l = r.sg_l;
    a.sg_h = r.sg_h;
    a.ts = ts;
    a.n_super = std::max(1, n_super_of(r.L, ts));
    a.n_prep = a.n_super;
    char *base = (char *)ws;
    if (a.n_super > 1) {
        a.wsS = (float *)(base + L.S);
        a.wsM = (float *)(base + L.M);
        a.wsN = (float *)(base + L.N);
        a.wsE = (float *)(base + L.E);
        a.wsDe = (float *)(base + L.De);
    }
    a.wsSc = (float *)(base + L.Sc);
    a.wsDc = (float *)(base + L.Dc);
    a.n_x = L.n_x;
    return gdn_run_bwd(a, r.D, (hipStream_t)stream, timing_of(tuning));
}

size_t sf_gdn_chain_workspace_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                                    const sf_tuning *tuning) {
    Shape r;
    GdnPlan p;
    if (resolve(shape, r) != SF_OK || check_segments(r, n_seg, seg_len) != SF_OK ||
        gdn_plan(r, n_seg, seg_len, tuning, p) != SF_OK)
        return 0;
    return gdn_chain_ws(r, p).total;
}

size_t sf_gdn_chain_ckpt_bytes(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len,
                               const sf_tuning *tuning) {
    g_err.clear();
    Shape r;
    GdnPlan p;
    if (resolve(shape, r) != SF_OK || check_segments(r, n_seg, seg_len) != SF_OK ||
        gdn_plan(r, n_seg, seg_len, tuning, p) != SF_OK)
        return 0;
    return gdn_ckpt_total(r, p);
}

sf_status sf_gdn_chain_fwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                           const void *k, const void *v, const float *g, const float *beta, void *o, float *S_bnd,
                           void *ckpt, size_t ckpt_bytes, void *v_new, void *ws, size_t ws_bytes,
                           const sf_tuning *tuning, sf_stream main_s, sf_stream aux_s) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    TRY(gdn_shape_ok(r));
    TRY(check_segments(r, n_seg, seg_len));
    if (!q || !k || !v || !g || !beta || !o || !S_bnd || !ws)
        return fail(SF_E_NULL, "q, k, v, g, beta, o, S_bnd and ws are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {o, "o"}, {S_bnd, "S_bnd"}, {ckpt, "ckpt"}, {v_new, "v_new"},
                     {ws, "ws"}}));
    if (((uintptr_t)g | (uintptr_t)beta) % 4) return fail(SF_E_ALIGN, "g and beta must be 4-byte aligned");
    GdnPlan p;
    TRY(gdn_plan(r, n_seg, seg_len, tuning, p));
    const GdnChainWs W = gdn_chain_ws(r, p);
    if (ws_bytes < W.total) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, W.total);
    const size_t kneed = gdn_ckpt_total(r, p);
    if (ckpt && ckpt_bytes < kneed) return fail(SF_E_WORKSPACE, "ckpt %zu < required %zu", ckpt_bytes, kneed);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"), grange(r, g, r.L, "g"),
                     grange(r, beta, r.L, "beta")},
                    {xrange(r, o, r.L, "o"), srange(r, S_bnd, n_seg + 1, "S_bnd"), xrange(r, v_new, r.L, "v_new"),
                     span(ckpt, (int64_t)kneed, "ckpt"), wsrange(ws, W.total)}));
    const int64_t SSB = (int64_t)r.B * r.H * r.D * r.D;
    const GdnFwdWs F = gdn_fwd_ws_n(r, p.n_max, p.n_max);
    std::vector<sf::GdnArgs> seg(n_seg);
    int64_t tok = 0;
    size_t kofs = 0;
    for (int i = 0; i < n_seg; ++i) {
        sf::GdnArgs &a = seg[i];
        a = gdn_seg_args(r, tok, seg_len[i], p.ts[i], q, k, v, g, beta);
        a.o = (void *)offset_x(r, o, tok);
        a.v_new = v_new ? (void *)offset_x(r, v_new, tok) : nullptr;
        a.S_in = S_bnd + i * SSB;
        a.S_out = S_bnd + (i + 1) * SSB;
        a.n_prep = a.n_super;  // maps of every superchunk: the scan writes S_out
        a.scan_out = 1;
        char *base = (char *)ws + (i % 2) * W.fwd_set;
        if (a.n_super > 1) {
            a.wsS = (float *)(base + F.S);
            a.wsM = (float *)(base + F.M);
            a.wsN = (float *)(base + F.N);
            if (ckpt) {  // S_J and M_J go to the kept-state buffer
                char *kb = (char *)ckpt + kofs;
                a.wsS = (float *)kb;
                a.wsM = (float *)(kb + gdn_ckpt_seg(r, a.n_super) / 2);
                kofs += gdn_ckpt_seg(r, a.n_super);
            }
        }
        tok += seg_len[i];
    }
    hipStream_t mn = (hipStream_t)main_s;
    hipStream_t ax = (aux_s && (!tuning || tuning->overlap != 0)) ? (hipStream_t)aux_s : mn;
    hipEvent_t e0 = nullptr, e1 = nullptr, sd[2] = {nullptr, nullptr};
    if (ax != mn) TRY(events(e0, e1, sd));
    // Schedule: Pre(i) on main -> ST(i) on aux, which also produces S_bnd[i+1],
    // so ST(i+1) follows ST(i) on aux while Out(i) runs on main after ST(i).
    // A single-superchunk segment's walk produces its S_out on main.  Out(i-1)
    // waits on main for ST(i-1), queued before Pre(i+1) overwrites workspace set
    // (i+1) % 2 = (i-1) % 2.
    int pending = -1;
    for (int i = 0; i < n_seg; ++i) {
        sf::GdnArgs &a = seg[i];
        if (a.n_super > 1) {
            TRY(gdn_launch(sf::GDN_PREP, a, r.D, mn, timing_of(tuning)));
            TRY(dep(mn, ax, e0));  // prep(i), and any S_bnd[i] written on main
            TRY(gdn_launch(sf::GDN_SCAN, a, r.D, ax, timing_of(tuning)));
            if (ax != mn) TRY(record(sd[i % 2], ax));
        }
        if (pending >= 0) {
            if (ax != mn) TRY(wait(mn, sd[pending % 2]));
            TRY(gdn_launch(sf::GDN_OUT, seg[pending], r.D, mn, timing_of(tuning)));
            pending = -1;
        }
        if (a.n_super > 1) {
            pending = i;
        } else {
            if (ax != mn && i > 0 && seg[i - 1].n_super > 1) TRY(wait(mn, sd[(i - 1) % 2]));  // S_bnd[i]
            TRY(gdn_launch(sf::GDN_OUT, a, r.D, mn, timing_of(tuning)));
        }
    }
    if (pending >= 0) {
        if (ax != mn) TRY(wait(mn, sd[pending % 2]));
        TRY(gdn_launch(sf::GDN_OUT, seg[pending], r.D, mn, timing_of(tuning)));
    }
    if (ax != mn) TRY(dep(ax, mn, e1));
    return SF_OK;
}

sf_status sf_gdn_chain_bwd(const sf_shape *shape, int32_t n_seg, const int64_t *seg_len, const void *q,
                           const void *k, const void *v, const float *g, const float *beta, const float *S_bnd,
                           const void *ckpt, size_t ckpt_bytes, const void *dO, const float *dS_final, void *dq,
                           void *dk, void *dv, float *dg, float *dbeta, float *dS_init, void *ws, size_t ws_bytes,
                           const sf_tuning *tuning, sf_stream main_s, sf_stream aux_s) {
    g_err.clear();
    Shape r;
    TRY(resolve(shape, r));
    TRY(check_timing(tuning));
    TRY(gdn_shape_ok(r));
    TRY(check_segments(r, n_seg, seg_len));
    if (!q || !k || !v || !g || !beta || !S_bnd || !dO || !dq || !dk || !dv || !dg || !dbeta || !dS_init || !ws)
        return fail(SF_E_NULL, "q, k, v, g, beta, S_bnd, dO, dq, dk, dv, dg, dbeta, dS_init and ws are required");
    TRY(check_align({{q, "q"}, {k, "k"}, {v, "v"}, {dO, "dO"}, {dq, "dq"}, {dk, "dk"}, {dv, "dv"}, {S_bnd, "S_bnd"},
                     {ckpt, "ckpt"}, {dS_final, "dS_final"}, {dS_init, "dS_init"}, {ws, "ws"}}));
    if (((uintptr_t)g | (uintptr_t)beta | (uintptr_t)dg | (uintptr_t)dbeta) % 4)
        return fail(SF_E_ALIGN, "g, beta, dg and dbeta must be 4-byte aligned");
    GdnPlan p;
    TRY(gdn_plan(r, n_seg, seg_len, tuning, p));
    const GdnChainWs W = gdn_chain_ws(r, p);
    if (ws_bytes < W.total) return fail(SF_E_WORKSPACE, "workspace %zu < required %zu", ws_bytes, W.total);
    const size_t kneed = gdn_ckpt_total(r, p);
    if (ckpt && ckpt_bytes < kneed) return fail(SF_E_WORKSPACE, "ckpt %zu < required %zu", ckpt_bytes, kneed);
    TRY(check_alias({xrange(r, q, r.L, "q"), xrange(r, k, r.L, "k"), xrange(r, v, r.L, "v"), grange(r, g, r.L, "g"),
                     grange(r, beta, r.L, "beta"), srange(r, S_bnd, n_seg, "S_bnd"), span(ckpt, (int64_t)kneed, "ckpt"),
                     xrange(r, dO, r.L, "dO"), srange(r, dS_final, 1, "dS_final")},
                    {xrange(r, dq, r.L, "dq"), xrange(r, dk, r.L, "dk"), xrange(r, dv, r.L, "dv"),
                     grange(r, dg, r.L, "dg"), grange(r, dbeta, r.L, "dbeta"), srange(r, dS_init, 1, "dS_init"),
                     wsrange(ws, W.total)}));
    const int64_t SSB = (int64_t)r.B * r.H * r.D * r.D;
    const GdnBwdWs Lw = gdn_bwd_ws_n(r, p.n_max, (size_t)p.nc_max);
    char *base = (char *)ws;
    float *dslot[2] = {(float *)(base + W.bwd), (float *)(base + W.bwd + W.dslot)};
    std::vector<sf::GdnArgs> seg(n_seg);
    std::vector<char> kept(n_seg, 0);
    int64_t tok = 0;
    size_t kofs = 0;
    for (int i = 0; i < n_seg; ++i) {
        sf::GdnArgs &a = seg[i];
        a = gdn_seg_args(r, tok, seg_len[i], p.ts[i], q, k, v, g, beta);
        a.S_in = S_bnd + i * SSB;
        a.dO = offset_x(r, dO, tok);
        a.dq = (void *)offset_x(r, dq, tok);
        a.dk = (void *)offset_x(r, dk, tok);
        a.dv = (void *)offset_x(r, dv, tok);
        a.dg = (float *)offset_g(r, dg, tok);
        a.dbeta = (float *)offset_g(r, dbeta, tok);
        // the state gradient leaving segment i enters it from segment i+1 (slot
        // (i+1) % 2), and the one entering goes to slot i % 2 (dS_init for i = 0)
        a.dS_out = i == n_seg - 1 ? dS_final : dslot[(i + 1) % 2];
        a.dS_in = i == 0 ? dS_init : dslot[i % 2];
        a.n_prep = a.n_super;
        if (a.n_super > 1) {
            a.wsS = (float *)(base + Lw.S);
            a.wsM = (float *)(base + Lw.M);
            a.wsN = (float *)(base + Lw.N);
            a.wsE = (float *)(base + Lw.E);
            a.wsDe = (float *)(base + Lw.De);
            if (ckpt) {  // the forward's S_J and M_J (read only)
                char *kb = (char *)ckpt + kofs;
                a.wsS = (float *)kb;
                a.wsM = (float *)(kb + gdn_ckpt_seg(r, a.n_super) / 2);
                kofs += gdn_ckpt_seg(r, a.n_super);
                kept[i] = 1;
            }
        }
        a.wsSc = (float *)(base + Lw.Sc);
        a.wsDc = (float *)(base + Lw.Dc);
        a.n_x = Lw.n_x;
        tok += seg_len[i];
    }
    hipStream_t mn = (hipStream_t)main_s;
    hipStream_t ax = (aux_s && (!tuning || tuning->overlap != 0)) ? (hipStream_t)aux_s : mn;
    hipEvent_t e0 = nullptr, e1 = nullptr, sd[2] = {nullptr, nullptr};
    if (ax != mn) TRY(events(e0, e1, sd));
    // Segments last to first.  Per segment on main: prep, dS prep, the
    // state-storing walk (after the scan), the dS walk (after the dS scan), the
    // per-chunk gradients; on aux: the scan after the prep (overlapping the dS
    // prep) and the dS scan after the dS prep and the next segment's dS walk
    // (overlapping the state-storing walk).  One workspace set serves every
    // segment: the next segment's prep follows this one's gradients on main,
    // and they follow both scans.
    for (int i = n_seg - 1; i >= 0; --i) {
        sf::GdnArgs &a = seg[i];
        if (a.n_super > 1) {
            if (!kept[i]) {  // replay the forward's maps and states
                TRY(gdn_launch(sf::GDN_PREP, a, r.D, mn, timing_of(tuning)));
                TRY(dep(mn, ax, e0));
                TRY(gdn_launch(sf::GDN_SCAN, a, r.D, ax, timing_of(tuning)));
                if (ax != mn) TRY(record(sd[0], ax));
            }
            TRY(gdn_launch(sf::GDN_DPREP, a, r.D, mn, timing_of(tuning)));
            TRY(dep(mn, ax, e1));  // dS prep, and dS_out written by the later segment's dS walk
            TRY(gdn_launch(sf::GDN_DSCAN, a, r.D, ax, timing_of(tuning)));
            if (ax != mn) {
                TRY(record(sd[1], ax));
                if (!kept[i]) TRY(wait(mn, sd[0]));
            }
        }
        TRY(gdn_launch(sf::GDN_STORE, a, r.D, mn, timing_of(tuning)));
        if (a.n_super > 1 && ax != mn) TRY(wait(mn, sd[1]));
        TRY(gdn_launch(sf::GDN_DWALK, a, r.D, mn, timing_of(tuning)));
        TRY(gdn_launch(sf::GDN_DCHUNK, a, r.D, mn, timing_of(tuning)));
    }
    return SF_OK;
}

sf_status sf_partition_hybrid(int64_t T, int32_t N, double alpha, double w_tok, double w_soft, int32_t round_to,
                              int64_t *seg_len) {
    g_err.clear();
    if (!seg_len) return fail(SF_E_NULL, "seg_len is NULL");
    if (T <= 0 || T > kPartMaxT || N < 1 || N > kPartMaxN || round_to < 1 || T % round_to)
        return fail(SF_E_SHAPE,
                    "need 0 < T <= 2^40 a multiple of round_to >= 1 and 1 <= N <= 2^20 (T=%lld N=%d round_to=%d)",
                    (long long)T, N, round_to);
    if (!(alpha >= 0.0) || !(w_tok >= 0.0) || !(w_soft >= 0.0) || !(w_tok + w_soft > 0.0) || !std::isfinite(alpha) ||
        !std::isfinite(w_tok) || !std::isfinite(w_soft))
        return fail(SF_E_SHAPE, "need alpha >= 0, w_tok >= 0, w_soft >= 0, not both weights 0");
    // accumulated cost A(c) = w_tok c + w_soft c^2 / 2 (Cost_i = A(c_{i+1}) - A(c_i));
    // the balanced boundary solves A(c) = (i / N) A(T), the positive root of a
    // quadratic, written in the cancellation-free form 2 r / (w_tok + sqrt(w_tok^2 + 2 w_soft r)).
    // That fp64 value is a first guess; the rounding is then decided exactly.
    const double Td = (double)T, total = w_tok * Td + 0.5 * w_soft * Td * Td;
    int64_t prev = 0;
    for (int32_t i = 1; i <= N; ++i) {
        int64_t c;
        if (i == N) {
            c = T;
        } else {
            const double r = total * (double)i / (double)N;
            const double hyb = 2.0 * r / (w_tok + std::sqrt(w_tok * w_tok + 2.0 * w_soft * r));
            const double equal = Td * (double)i / (double)N;
            const double x = (1.0 - alpha) * equal + alpha * hyb;
            // closest multiple of round_to, half-way cases up: the largest m
            // in [0, T / R] with c_i >= (m - 1/2) R, decided exactly; the fp64
            // value is tried first, else a binary search (it may be inf or NaN
            // for extreme weights)
            const int64_t top = T / round_to;
            auto ok = [&](int64_t m) {
                return m == 0 || part_at_least(T, N, i, alpha, w_tok, w_soft, round_to, 2 * m - 1);
            };
            int64_t m = -1;
            if (std::isfinite(x) && x > -(double)round_to && x < (double)T + round_to) {
                const int64_t g = std::max<int64_t>(0, std::min<int64_t>((int64_t)std::floor(x / round_to + 0.5), top));
                if (ok(g) && (g == top || !ok(g + 1))) m = g;
            }
            if (m < 0) {
                int64_t lo = 0, hi = top;  // ok(lo) holds
                while (lo < hi) {
                    const int64_t mid = lo + (hi - lo + 1) / 2;
                    if (ok(mid)) lo = mid;
                    else hi = mid - 1;
                }
                m = lo;
            }
            c = m * round_to;
        }
        if (c <= prev || c > T)
            return fail(SF_E_SHAPE, "segment %d is empty or out of range after rounding (boundary %lld)", i - 1,
                        (long long)c);
        seg_len[i - 1] = c - prev;
        prev = c;
    }
    return SF_OK;
}

}  // extern "C"
