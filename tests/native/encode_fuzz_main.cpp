// Standalone round-trip driver for the host encoder/decoder, built with
// AddressSanitizer and UBSan by the CPU test suite. Random shapes, densities
// and bit patterns; every decode must equal the masked input bit for bit.
#include <cstdio>
#include <random>
#include <vector>

#include "../../paper_2607_08786_amd/csrc/usp_internal.h"

int main() {
    std::mt19937_64 rng(12345);
    for (int it = 0; it < 60; ++it) {
        const int64_t M = 1 + (int64_t)(rng() % 70), K = 1 + (int64_t)(rng() % 700);
        const int64_t ldw = K + (int64_t)(rng() % 3), ldm = K + (int64_t)(rng() % 5);
        const double d = (rng() % 101) / 100.0;
        std::vector<uint16_t> W((size_t)(M * ldw));
        std::vector<uint8_t> mask((size_t)(M * ldm));
        for (auto &w : W) w = (uint16_t)rng();
        std::uniform_real_distribution<double> u(0.0, 1.0);
        for (auto &m : mask) m = u(rng) < d ? (uint8_t)(1 + rng() % 255) : 0;
        usp::HostEncoding enc;
        usp::encode_host(W.data(), ldw, mask.data(), ldm, M, K, enc);
        std::vector<uint16_t> Wo((size_t)(M * K));
        std::vector<uint8_t> mo((size_t)(M * K));
        if (!usp::decode_host(enc, Wo.data(), mo.data())) { std::printf("decode failed\n"); return 1; }
        for (int64_t m = 0; m < M; ++m)
            for (int64_t k = 0; k < K; ++k) {
                const bool kept = mask[m * ldm + k] != 0;
                if (mo[m * K + k] != (kept ? 1 : 0) || Wo[m * K + k] != (kept ? W[m * ldw + k] : 0)) {
                    std::printf("mismatch it=%d m=%ld k=%ld\n", it, (long)m, (long)k);
                    return 1;
                }
            }
    }
    std::printf("ok\n");
    return 0;
}
