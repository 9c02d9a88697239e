// Host-only harness around the library's encoder/decoder (usp_encode.cpp), so
// that the CPU test suite can check the format without a GPU.
#include <cstring>
#include <new>

#include "../../paper_2607_08786_amd/csrc/usp_internal.h"

extern "C" {

// Encodes, reports sizes, decodes back. Returns 0 on success.
int usp_test_roundtrip(const uint16_t *W, int64_t ldw, const uint8_t *mask, int64_t ldm, int64_t M, int64_t K,
                       uint16_t *W_out, uint8_t *mask_out, int64_t *nnz, int64_t *stream_bytes,
                       int64_t *tiles) {
    usp::HostEncoding enc;
    try {
        usp::encode_host(W, ldw, mask, ldm, M, K, enc);
    } catch (const std::bad_alloc &) {
        return 1;
    }
    *nnz = enc.nnz;
    *stream_bytes = (int64_t)enc.stream.size();
    *tiles = enc.RB * enc.KT;
    return usp::decode_host(enc, W_out, mask_out) ? 0 : 2;
}

// Copies the raw records and offset table (caller sizes them from a first call).
int usp_test_records(const uint16_t *W, const uint8_t *mask, int64_t M, int64_t K, uint8_t *stream_out,
                     uint32_t *off_out) {
    usp::HostEncoding enc;
    usp::encode_host(W, K, mask, K, M, K, enc);
    std::memcpy(stream_out, enc.stream.data(), enc.stream.size());
    std::memcpy(off_out, enc.off.data(), enc.off.size() * sizeof(uint32_t));
    return 0;
}
}
