// Host-side ABI checks run under AddressSanitizer and UndefinedBehaviorSanitizer:
// argument validation of every entry point (fake device pointers that are never
// dereferenced; the launch stubs abort if anything is launched) and the
// hybrid-aware partition, whose exact rounding runs big-integer arithmetic.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "stateflow.h"

static int failures = 0;
#define EXPECT(cond)                                                        \
    do {                                                                    \
        if (!(cond)) {                                                      \
            std::fprintf(stderr, "%s:%d: FAILED %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                     \
        }                                                                   \
    } while (0)

static void *P(int i) { return (void *)(uintptr_t)(0x7F0000000000ull + (uint64_t)i * (1ull << 32)); }
static float *F(int i) { return (float *)P(i); }

static sf_shape shape(int64_t L = 1024) {
    sf_shape s;
    std::memset(&s, 0, sizeof s);
    s.B = 1, s.H = 2, s.Dk = 128, s.Dv = 128, s.L = L, s.chunk = 64, s.io_dtype = SF_BF16, s.gate = SF_GATE_SCALAR;
    return s;
}

int main() {
    sf_tuning t;
    std::memset(&t, 0, sizeof t);
    t.ts = 128;
    sf_shape s = shape();
    // segment forward
    EXPECT(sf_segment_fwd(nullptr, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_NULL);
    sf_shape bad = shape(100);
    EXPECT(sf_segment_fwd(&bad, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_SHAPE);
    bad = shape();
    bad.Dk = 96, bad.Dv = 96;
    EXPECT(sf_segment_fwd(&bad, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) ==
           SF_E_UNSUPPORTED);
    bad = shape();
    bad.io_dtype = 7;
    EXPECT(sf_segment_fwd(&bad, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_DTYPE);
    EXPECT(sf_segment_fwd(&s, (char *)P(1) + 2, P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) ==
           SF_E_ALIGN);
    EXPECT(sf_segment_fwd(&s, P(1), P(2), P(3), F(4), nullptr, P(1), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_ALIAS);
    EXPECT(sf_segment_fwd(&s, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(5), 1 << 30, &t, nullptr) == SF_E_ALIAS);
    EXPECT(sf_segment_fwd(&s, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 16, &t, nullptr) == SF_E_WORKSPACE);
    EXPECT(std::strlen(sf_last_error()) > 0);
    // segment backward
    EXPECT(sf_segment_bwd(&s, P(1), P(2), P(3), F(4), nullptr, P(6), nullptr, P(8), P(9), P(10), F(11), F(12), P(8),
                          1 << 30, &t, nullptr) == SF_E_ALIAS);
    EXPECT(sf_segment_bwd(&s, P(1), P(2), P(3), F(4), nullptr, P(6), nullptr, P(8), P(9), P(10), F(11), nullptr,
                          P(13), 1 << 30, &t, nullptr) == SF_E_NULL);
    // chains
    const int64_t segs[2] = {512, 448};
    EXPECT(sf_chain_fwd(&s, 2, segs, P(1), P(2), P(3), F(4), P(5), F(6), nullptr, 0, P(7), 1 << 30, nullptr, nullptr, nullptr) ==
           SF_E_SHAPE);
    const int64_t segs2[2] = {512, 512};
    EXPECT(sf_chain_fwd(&s, 2, segs2, P(1), P(2), P(3), F(4), P(5), F(6), nullptr, 0, P(5), 1 << 30, nullptr, nullptr, nullptr) ==
           SF_E_ALIAS);
    EXPECT(sf_chain_bwd(&s, 2, segs2, P(1), P(2), P(3), F(4), F(5), nullptr, 0, P(6), nullptr, P(8), P(9), P(10), F(11), nullptr,
                        P(13), 1 << 30, nullptr, nullptr, nullptr) == SF_E_NULL);
    EXPECT(sf_chain_workspace_bytes(&s, 2, segs2, nullptr) > 0);
    EXPECT(sf_chain_workspace_bytes(&s, 2, segs, nullptr) == 0);
    // kept superchunk states
    sf_tuning t128;
    std::memset(&t128, 0, sizeof t128);
    t128.ts = 128;
    const size_t kneed = sf_chain_ckpt_bytes(&s, 2, segs2, &t128);
    EXPECT(kneed > 0);
    EXPECT(sf_chain_ckpt_bytes(&s, 2, segs, &t128) == 0 && std::strlen(sf_last_error()) > 0);
    EXPECT(sf_chain_fwd(&s, 2, segs2, P(1), P(2), P(3), F(4), P(5), F(6), P(8), kneed - 1, P(7), 1 << 30, &t128,
                        nullptr, nullptr) == SF_E_WORKSPACE);
    EXPECT(sf_chain_bwd(&s, 2, segs2, P(1), P(2), P(3), F(4), F(5), P(8), kneed, P(6), nullptr, P(8), P(9), P(10),
                        F(11), F(12), P(13), 1 << 30, &t128, nullptr, nullptr) == SF_E_ALIAS);
    // timing record
    sf_timing tm;
    std::memset(&tm, 0, sizeof tm);
    tm.capacity = 4, tm.count = 5;
    t.timing = &tm;
    EXPECT(sf_segment_fwd(&s, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_SHAPE);
    tm.count = 0;
    EXPECT(sf_segment_fwd(&s, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), P(7), 1 << 30, &t, nullptr) == SF_E_NULL);
    t.timing = nullptr;
    // allocation-free forward: oversized shapes are rejected before any launch
    sf_shape big = shape(65536);
    big.H = 40;
    sf_tuning t64;
    std::memset(&t64, 0, sizeof t64);
    t64.ts = 64;
    EXPECT(sf_segment_fwd_noalloc(&big, P(1), P(2), P(3), F(4), nullptr, P(5), F(6), &t64, nullptr) == SF_E_WORKSPACE);
    // short convolution
    sf_conv_shape c;
    std::memset(&c, 0, sizeof c);
    c.B = 2, c.C = 64, c.L = 1000, c.W = 4, c.io_dtype = SF_BF16, c.act = SF_ACT_SILU;
    EXPECT(sf_conv_fwd(&c, P(1), F(2), F(3), P(1), F(5), nullptr, nullptr) == SF_E_ALIAS);
    c.C = 12;
    EXPECT(sf_conv_fwd(&c, P(1), F(2), F(3), P(4), F(5), nullptr, nullptr) == SF_E_UNSUPPORTED);
    c.C = 64;
    EXPECT(sf_conv_bwd(&c, P(1), F(2), F(3), P(4), F(5), P(6), F(7), F(8), P(9), 16, nullptr, nullptr) ==
           SF_E_WORKSPACE);
    // gated delta rule
    EXPECT(sf_gdn_fwd(&s, P(1), P(2), P(3), F(4), F(5), nullptr, P(1), F(7), nullptr, P(8), 1ull << 40, nullptr,
                      nullptr) == SF_E_ALIAS);
    EXPECT(sf_gdn_bwd(&s, P(1), P(2), P(3), F(4), F(5), nullptr, P(6), nullptr, P(7), P(8), P(9), F(10), F(11), F(12),
                      P(7), 1ull << 40, nullptr, nullptr) == SF_E_ALIAS);
    EXPECT(sf_gdn_chain_fwd(&s, 2, segs2, P(1), P(2), P(3), F(4), F(5), P(1), F(7), nullptr, 0, nullptr, P(8),
                            1ull << 40, nullptr, nullptr, nullptr) == SF_E_ALIAS);
    const size_t gk = sf_gdn_chain_ckpt_bytes(&s, 2, segs2, &t128);
    EXPECT(gk > 0);
    EXPECT(sf_gdn_chain_fwd(&s, 2, segs2, P(1), P(2), P(3), F(4), F(5), P(6), F(7), P(9), gk - 1, nullptr, P(8),
                            1ull << 40, &t128, nullptr, nullptr) == SF_E_WORKSPACE);
    EXPECT(sf_gdn_chain_bwd(&s, 2, segs2, P(1), P(2), P(3), F(4), F(5), F(7), P(9), gk, P(6), nullptr, P(9), P(10),
                            P(11), F(12), F(13), F(14), P(8), 1ull << 40, &t128, nullptr, nullptr) == SF_E_ALIAS);
    // partition: exact half-way cases round up, irrational boundaries, errors
    int64_t len[8];
    EXPECT(sf_partition_hybrid(384, 2, 0.0, 1.0, 1.0, 128, len) == SF_OK && len[0] == 256 && len[1] == 128);
    EXPECT(sf_partition_hybrid(384, 2, 1.25, 1.0, 0.0, 128, len) == SF_OK && len[0] == 256 && len[1] == 128);
    EXPECT(sf_partition_hybrid(1280, 4, 1.0, 0.0, 1.0, 128, len) == SF_OK && len[0] == 640 && len[1] == 256 &&
           len[2] == 256 && len[3] == 128);
    EXPECT(sf_partition_hybrid(640, 4, 1.0, 0.0, 1e-3, 128, len) == SF_E_SHAPE);
    EXPECT(sf_partition_hybrid(262144, 8, 1.0, 1e-300, 1e300, 128, len) == SF_OK);  // wide exponent gaps
    EXPECT(sf_partition_hybrid(262144, 8, 0.7, 7.5, 4.9e-324, 64, len) == SF_OK);   // a subnormal weight
    EXPECT(sf_partition_hybrid(int64_t(1) << 41, 8, 1.0, 1.0, 0.0, 128, len) == SF_E_SHAPE);
    EXPECT(sf_partition_hybrid(262144, 8, 1.0, 1.0, 1e-5, 128, nullptr) == SF_E_NULL);
    if (failures) std::fprintf(stderr, "%d check(s) failed\n", failures);
    else std::printf("abi checks passed\n");
    return failures ? 1 : 0;
}
