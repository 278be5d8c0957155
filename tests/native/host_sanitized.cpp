// Drives the host-only library functions (cache plan, expert packers, error reporting)
// over random and invalid inputs, built with AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_host_sanitized.py: every buffer is exactly as large as the declarations in
// apex.h say, so an access past it, or undefined behaviour inside, stops the program.
// Prints "ok" when every check passed.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "apex.h"

namespace {

int failures = 0;

void check(bool ok, const char *what) {
    if (!ok) {
        std::printf("FAIL: %s\n", what);
        ++failures;
    }
}

uint16_t bf16_bits(float f) {
    uint32_t u;
    std::memcpy(&u, &f, sizeof u);
    return uint16_t((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// finite bf16 values of every kind: zeros of both signs, subnormals, ordinary values and
// the largest finite magnitudes
std::vector<uint16_t> weights(std::mt19937 &rng, size_t n) {
    std::vector<uint16_t> w(n);
    std::normal_distribution<float> nd(0.f, 0.02f);
    std::uniform_int_distribution<int> kind(0, 19);
    for (auto &v : w) {
        switch (kind(rng)) {
            case 0: v = 0x0000; break;
            case 1: v = 0x8000; break;
            case 2: v = uint16_t(0x0001 + rng() % 0x7f); break;   // subnormal
            case 3: v = 0x7f7f; break;                             // largest finite
            case 4: v = 0xff7f; break;
            default: v = bf16_bits(nd(rng));
        }
    }
    return w;
}

void plans(std::mt19937 &rng) {
    for (int trial = 0; trial < 400; ++trial) {
        const int E = 1 + int(rng() % 64);
        const int C = 1 + int(rng() % E);
        const int k_max = 1 + int(rng() % C);
        const int B = int(rng() % 9);
        std::vector<int32_t> eos(C);
        for (int s = 0; s < C; ++s) eos[s] = (s < E && rng() % 4) ? s : -1;
        std::vector<int64_t> last_used(E, -1);
        for (int64_t step = 0; step < 12; ++step) {
            std::vector<int32_t> pf_idx(size_t(B) * k_max, -1), pf_count(B);
            for (int b = 0; b < B; ++b) {
                std::vector<int32_t> perm(E);
                for (int e = 0; e < E; ++e) perm[e] = e;
                std::shuffle(perm.begin(), perm.end(), rng);
                pf_count[b] = int32_t(rng() % (k_max + 1));
                for (int j = 0; j < pf_count[b]; ++j) pf_idx[size_t(b) * k_max + j] = perm[j];
            }
            std::vector<int32_t> ce(C), cs(C);
            int n = -1;
            const apex_status st =
                apex_plan_residency(E, C, B ? pf_idx.data() : nullptr,
                                    B ? pf_count.data() : nullptr, B, k_max, step, eos.data(),
                                    last_used.data(), ce.data(), cs.data(), &n);
            check(st == APEX_OK && n >= 0 && n <= C, "plan on valid input");
            // every copied expert sits in the slot it was copied to, once
            std::vector<int> seen(E, 0);
            for (int s = 0; s < C; ++s)
                if (eos[s] >= 0) seen[eos[s]] += 1;
            for (int e = 0; e < E; ++e) check(seen[e] <= 1, "an expert in two slots");
            for (int i = 0; i < n; ++i) check(eos[cs[i]] == ce[i], "copy lands in its slot");
        }
        // invalid sets and states: refused, nothing written
        if (B > 0) {
            std::vector<int32_t> pf_idx(size_t(B) * k_max, 0), pf_count(B, 1);
            pf_idx[0] = E;                                  // expert id out of range
            std::vector<int32_t> before = eos, ce(C), cs(C);
            int n = 0;
            check(apex_plan_residency(E, C, pf_idx.data(), pf_count.data(), B, k_max, 99,
                                      eos.data(), last_used.data(), ce.data(), cs.data(),
                                      &n) == APEX_E_INVAL,
                  "out-of-range expert refused");
            check(eos == before, "refused plan leaves the state");
            check(std::strlen(apex_last_error()) > 0, "error message set");
            pf_idx[0] = 0;
            pf_count[0] = k_max + 1;                         // set longer than k_max
            check(apex_plan_residency(E, C, pf_idx.data(), pf_count.data(), B, k_max, 99,
                                      eos.data(), last_used.data(), ce.data(), cs.data(),
                                      &n) == APEX_E_INVAL,
                  "overlong set refused");
        }
        if (C >= 2 && E >= 1) {
            std::vector<int32_t> dup(C, -1), ce(C), cs(C);
            dup[0] = dup[1] = 0;                             // expert 0 in two slots
            int n = 0;
            check(apex_plan_residency(E, C, nullptr, nullptr, 0, k_max, 0, dup.data(),
                                      last_used.data(), ce.data(), cs.data(), &n) ==
                      APEX_E_INVAL,
                  "repeated expert refused");
        }
    }
    int n = 0;
    check(apex_plan_residency(65, 4, nullptr, nullptr, 0, 1, 0, nullptr, nullptr, nullptr,
                              nullptr, &n) == APEX_E_INVAL,
          "E above 64 refused");
}

void packers(std::mt19937 &rng) {
    const int shapes[][2] = {{32, 32}, {64, 96}, {256, 64}, {96, 160}, {512, 32}};
    for (const auto &sh : shapes) {
        const int d = sh[0], I = sh[1];
        const size_t n = size_t(d) * I;
        const auto w1 = weights(rng, n), w3 = weights(rng, n), w2 = weights(rng, n);
        {
            std::vector<uint16_t> out(apex_expert_bytes(d, I) / 2);
            check(apex_pack_expert(w1.data(), w3.data(), w2.data(), d, I, out.data()) ==
                      APEX_OK,
                  "bf16 pack");
            check(out[1] == w1[1] && out[d] == w3[0] && out[2 * n] == w2[0], "bf16 layout");
        }
        {
            std::vector<uint8_t> out(apex_expert_bytes_fp8(d, I));
            check(apex_pack_expert_fp8(w1.data(), w3.data(), w2.data(), d, I, out.data()) ==
                      APEX_OK,
                  "fp8 pack");
            float s;   // the scales are finite and non-negative
            for (size_t r = 0; r < size_t(2 * I + d); ++r) {
                std::memcpy(&s, out.data() + 3 * n + 4 * r, 4);
                check(std::isfinite(s) && s >= 0.f, "fp8 scale finite");
            }
        }
        {
            std::vector<uint8_t> out(apex_expert_bytes_mxfp4(d, I));
            check(apex_pack_expert_mxfp4(w1.data(), w3.data(), w2.data(), d, I, out.data()) ==
                      APEX_OK,
                  "mxfp4 pack");
        }
        {
            std::vector<float> out(apex_expert_bytes_fp32(d, I) / 4);
            check(apex_pack_expert_fp32(w1.data(), w3.data(), w2.data(), d, I, out.data()) ==
                      APEX_OK,
                  "fp32 pack");
        }
    }
    // shapes the formats cannot hold, and NULL buffers: refused before any write
    std::vector<uint16_t> w(64 * 48, 0);
    std::vector<uint8_t> out(1 << 16);
    check(apex_pack_expert_fp8(w.data(), w.data(), w.data(), 64, 12, out.data()) ==
              APEX_E_INVAL,
          "fp8 I not a multiple of 8");
    check(apex_pack_expert_mxfp4(w.data(), w.data(), w.data(), 64, 48, out.data()) ==
              APEX_E_INVAL,
          "mxfp4 I not a multiple of 32");
    check(apex_pack_expert_fp32(w.data(), w.data(), w.data(), 64, 6, out.data()) ==
              APEX_E_INVAL,
          "fp32 I not a multiple of 4");
    check(apex_pack_expert(nullptr, w.data(), w.data(), 8, 8,
                           reinterpret_cast<uint16_t *>(out.data())) == APEX_E_INVAL,
          "bf16 NULL input");
    check(apex_expert_bytes(0, 8) == 0 && apex_expert_bytes_fp8(8, -1) == 0 &&
              apex_expert_bytes_mxfp4(-32, 32) == 0 && apex_expert_bytes_fp32(0, 0) == 0,
          "sizes of empty shapes");
}

}  // namespace

int main() {
    std::mt19937 rng(20261202);
    plans(rng);
    packers(rng);
    if (failures) {
        std::printf("%d failures\n", failures);
        return 1;
    }
    std::printf("ok\n");
    return 0;
}
