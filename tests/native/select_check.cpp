// Host-only check of the top-k selection's key and radix-digit schedule
// (sel_mag, sel_key, kSelTopShift, sel_next_shift from ts_plan.h, the same
// constexpr definitions the selection kernels use).  A host model of the
// kernels' steps (a 256-bin histogram per digit over the keys matching the
// prefix found so far, the bin holding the remaining rank counted from the
// top, the early stop when the whole bin is kept, the tie-break over
// 0xffff - neuron index) must keep exactly the `keep` largest magnitudes,
// ties to the lower index, as a sort does.  Inputs include negative values,
// -0, infinities, NaN patterns and many exact ties.  Built with g++ and the
// sanitizers by tests/test_plan_cpu.py; prints "ok" or the first failure.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "ts_plan.h"

using namespace ts;

namespace {

// The bin holding the rem-th largest counted key: returns the digit, sets
// rem to the rank left inside the bin and cnt to the bin's count.
int find_bin(const uint32_t (&hist)[256], uint32_t &rem, uint32_t &cnt) {
    uint32_t above = 0;
    for (int b = 255; b >= 0; --b) {
        if (above + hist[b] >= rem) {
            rem -= above;
            cnt = hist[b];
            return b;
        }
        above += hist[b];
    }
    return -1;
}

// Kept flags of the model (keys as the selection kernel forms them).
std::vector<bool> model_keep(const std::vector<uint32_t> &bits, const std::vector<int> &idx, int keep, bool *bad) {
    const int n = (int)bits.size();
    std::vector<uint32_t> key(n);
    for (int i = 0; i < n; ++i) {
        key[i] = sel_key(bits[i]);
        if (key[i] >> 31) *bad = true;  // the first digit must stay below 256
    }
    const int k = std::min(keep, n);
    uint32_t thr = 0xffffffffu, tie_n = 0xffffu;
    if (k > 0) {
        uint32_t prefix = 0, mask = 0, rem = (uint32_t)k, cnt = 0;
        for (int shift = kSelTopShift; shift >= 0; shift = sel_next_shift(shift)) {
            uint32_t hist[256] = {};
            for (int i = 0; i < n; ++i)
                if ((key[i] & mask) == prefix) {
                    const uint32_t b = key[i] >> shift;
                    if (shift == kSelTopShift && b > 255u) *bad = true;
                    ++hist[b & 255u];
                }
            const int d = find_bin(hist, rem, cnt);
            if (d < 0) {
                *bad = true;
                return {};
            }
            prefix |= (uint32_t)d << shift;
            mask |= 255u << shift;
            if (rem == cnt) break;  // the whole bin kept: its floor is the threshold
        }
        thr = prefix;
        if (rem < cnt) {  // only some keys equal to thr kept: the rem-th smallest index
            uint32_t p2 = 0, m2 = 0, r2 = rem, c2 = 0;
            for (int shift = 8; shift >= 0; shift -= 8) {
                uint32_t hist[256] = {};
                for (int i = 0; i < n; ++i) {
                    const uint32_t q = 0xffffu - (uint32_t)idx[i];
                    if (key[i] == thr && (q & m2) == p2) ++hist[(q >> shift) & 255u];
                }
                const int d = find_bin(hist, r2, c2);
                if (d < 0) {
                    *bad = true;
                    return {};
                }
                p2 |= (uint32_t)d << shift;
                m2 |= 255u << shift;
            }
            tie_n = 0xffffu - p2;
        }
    }
    std::vector<bool> kept(n);
    for (int i = 0; i < n; ++i) kept[i] = key[i] > thr || (key[i] == thr && (uint32_t)idx[i] <= tie_n);
    return kept;
}

// Reference: sort by magnitude descending (NaN as +inf), then index ascending.
std::vector<bool> sort_keep(const std::vector<uint32_t> &bits, const std::vector<int> &idx, int keep) {
    const int n = (int)bits.size();
    auto mag = [&](int i) {
        float f;
        std::memcpy(&f, &bits[i], 4);
        f = std::fabs(f);
        return f != f ? __builtin_inff() : f;
    };
    std::vector<int> ord(n);
    for (int i = 0; i < n; ++i) ord[i] = i;
    std::sort(ord.begin(), ord.end(), [&](int a, int b) {
        const float ma = mag(a), mb = mag(b);
        return ma != mb ? ma > mb : idx[a] < idx[b];
    });
    std::vector<bool> kept(n, false);
    for (int j = 0; j < std::min(keep, n); ++j) kept[ord[j]] = true;
    return kept;
}

uint32_t f2u(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

}  // namespace

int main() {
    // the schedule: 23, 15, 7, 0, then done; every bit 0..30 covered
    int shifts[8], ns = 0;
    for (int s = kSelTopShift; s >= 0 && ns < 8; s = sel_next_shift(s)) shifts[ns++] = s;
    if (ns != 4 || shifts[0] != 23 || shifts[1] != 15 || shifts[2] != 7 || shifts[3] != 0) {
        std::printf("FAIL schedule\n");
        return 1;
    }
    uint32_t covered = 0;
    for (int i = 0; i < ns; ++i) covered |= 255u << shifts[i];
    if (covered != 0x7fffffffu) {
        std::printf("FAIL coverage %08x\n", covered);
        return 1;
    }
    // keys: sign cleared, NaN clamped, +1
    if (sel_key(f2u(-2.5f)) != f2u(2.5f) + 1u || sel_key(f2u(-0.0f)) != 1u || sel_key(0xffffffffu) != 0x7f800001u ||
        sel_key(0x7fc00000u) != 0x7f800001u || sel_mag(f2u(-1.0f)) != f2u(1.0f)) {
        std::printf("FAIL keys\n");
        return 1;
    }

    std::mt19937_64 rng(12345);
    std::normal_distribution<float> nd(0.f, 1.f);
    for (int trial = 0; trial < 3000; ++trial) {
        const int n = 1 + (int)(rng() % 700);
        std::vector<uint32_t> bits(n);
        std::vector<int> idx(n);
        const int mode = trial % 6;
        for (int i = 0; i < n; ++i) {
            float v = nd(rng);
            if (mode == 0) v = std::fabs(v);                         // dReLU values
            if (mode == 2) v = (float)(int)(rng() % 5) * 0.25f;      // many exact ties, zeros
            if (mode == 3) v = std::ldexp(1.0f, (int)(rng() % 40) - 20);  // one bin per octave
            bits[i] = f2u(v);
            if (mode == 4 && rng() % 17 == 0) bits[i] = (rng() & 1) ? 0x7f800000u : 0xff800000u;  // +-inf
            if (mode == 5 && rng() % 23 == 0) bits[i] = 0x7fc00000u | (uint32_t)(rng() & 1) << 31;  // NaN
            if (mode == 5 && rng() % 29 == 0) bits[i] = 0x80000000u;                                // -0
        }
        // neuron indices: distinct, not in list order (interleaved tiles)
        for (int i = 0; i < n; ++i) idx[i] = i;
        std::shuffle(idx.begin(), idx.end(), rng);
        const int keeps[] = {0, 1, n / 10, n / 2, n - 1, n, n + 5, 1 + (int)(rng() % n)};
        for (int keep : keeps) {
            if (keep < 0) continue;
            bool bad = false;
            const std::vector<bool> got = model_keep(bits, idx, keep, &bad);
            const std::vector<bool> want = sort_keep(bits, idx, keep);
            if (bad || got != want) {
                std::printf("FAIL trial %d mode %d n %d keep %d\n", trial, mode, n, keep);
                return 1;
            }
        }
    }
    std::printf("ok\n");
    return 0;
}
