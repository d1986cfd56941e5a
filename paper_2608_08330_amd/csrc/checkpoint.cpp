// Weights checkpoint parsing and verification, and the SHA-256 it uses.
#include "checkpoint.hpp"

#include <array>
#include <cstring>

namespace rtcc {

namespace {

// ---------------------------------------------------------------------------
// SHA-256 (FIPS 180-4).  The round constants are the first 32 bits of the
// fractional parts of the cube roots of the first 64 primes, the initial
// hash the same of the square roots of the first 8 primes; both are computed
// here exactly with integer roots: floor(cbrt(p * 2^96)) and
// floor(sqrt(p * 2^64)) keep the integer part above bit 32, so their low 32
// bits are those fractional bits.
// ---------------------------------------------------------------------------

using u128 = unsigned __int128;

uint64_t int_root(u128 x, int degree) {
    // largest y with y^degree <= x (y < 2^40 for the arguments used here)
    uint64_t lo = 0, hi = uint64_t(1) << 40;
    while (hi - lo > 1) {
        const uint64_t mid = lo + (hi - lo) / 2;
        u128 pw = 1;
        for (int i = 0; i < degree; ++i) pw *= mid;
        if (pw <= x) lo = mid; else hi = mid;
    }
    return lo;
}

struct ShaConstants {
    uint32_t k[64];
    uint32_t h0[8];
    ShaConstants() {
        int found = 0;
        for (uint32_t p = 2; found < 64; ++p) {
            bool prime = true;
            for (uint32_t d = 2; d * d <= p; ++d)
                if (p % d == 0) { prime = false; break; }
            if (!prime) continue;
            k[found] = uint32_t(int_root(u128(p) << 96, 3));
            if (found < 8) h0[found] = uint32_t(int_root(u128(p) << 64, 2));
            ++found;
        }
    }
};

const ShaConstants &sha_constants() {
    static const ShaConstants c;
    return c;
}

inline uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

void sha_block(uint32_t h[8], const unsigned char *b, const uint32_t k[64]) {
    uint32_t w[64];
    for (int t = 0; t < 16; ++t)
        w[t] = uint32_t(b[4 * t]) << 24 | uint32_t(b[4 * t + 1]) << 16 | uint32_t(b[4 * t + 2]) << 8 | b[4 * t + 3];
    for (int t = 16; t < 64; ++t) {
        const uint32_t s0 = rotr(w[t - 15], 7) ^ rotr(w[t - 15], 18) ^ (w[t - 15] >> 3);
        const uint32_t s1 = rotr(w[t - 2], 17) ^ rotr(w[t - 2], 19) ^ (w[t - 2] >> 10);
        w[t] = s1 + w[t - 7] + s0 + w[t - 16];
    }
    uint32_t a = h[0], bb = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], hh = h[7];
    for (int t = 0; t < 64; ++t) {
        const uint32_t big1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
        const uint32_t ch = (e & f) ^ (~e & g);
        const uint32_t t1 = hh + big1 + ch + k[t] + w[t];
        const uint32_t big0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
        const uint32_t maj = (a & bb) ^ (a & c) ^ (bb & c);
        const uint32_t t2 = big0 + maj;
        hh = g; g = f; f = e; e = d + t1; d = c; c = bb; bb = a; a = t1 + t2;
    }
    h[0] += a; h[1] += bb; h[2] += c; h[3] += d; h[4] += e; h[5] += f; h[6] += g; h[7] += hh;
}

// little-endian field readers (the checkpoint is little endian on every host)
uint32_t rd32(const unsigned char *p) {
    return uint32_t(p[0]) | uint32_t(p[1]) << 8 | uint32_t(p[2]) << 16 | uint32_t(p[3]) << 24;
}
uint64_t rd64(const unsigned char *p) { return uint64_t(rd32(p)) | uint64_t(rd32(p + 4)) << 32; }

bool nul_terminated(const unsigned char *p, size_t n, std::string &out) {
    for (size_t i = 0; i < n; ++i)
        if (p[i] == 0) {
            out.assign(reinterpret_cast<const char *>(p), i);
            for (size_t j = i; j < n; ++j)
                if (p[j] != 0) return false;  // padding must be zero
            return true;
        }
    return false;
}

const char kMagic[8] = {'R', 'T', 'C', 'C', 'W', 'G', 'T', '\0'};

}  // namespace

void sha256(const void *data, size_t n, uint8_t out[32]) {
    const ShaConstants &c = sha_constants();
    uint32_t h[8];
    std::memcpy(h, c.h0, sizeof(h));
    const unsigned char *p = static_cast<const unsigned char *>(data);
    size_t full = n / 64;
    for (size_t i = 0; i < full; ++i) sha_block(h, p + 64 * i, c.k);
    // padding: 0x80, zeros up to 56 mod 64, then the bit length big endian
    unsigned char tail[128] = {};
    const size_t rem = n - 64 * full;
    if (rem) std::memcpy(tail, p + 64 * full, rem);
    tail[rem] = 0x80;
    const size_t tail_len = rem + 1 + 8 <= 64 ? 64 : 128;
    const uint64_t bits = uint64_t(n) * 8;
    for (int i = 0; i < 8; ++i) tail[tail_len - 1 - i] = uint8_t(bits >> (8 * i));
    for (size_t off = 0; off < tail_len; off += 64) sha_block(h, tail + off, c.k);
    for (int i = 0; i < 8; ++i) {
        out[4 * i] = uint8_t(h[i] >> 24);
        out[4 * i + 1] = uint8_t(h[i] >> 16);
        out[4 * i + 2] = uint8_t(h[i] >> 8);
        out[4 * i + 3] = uint8_t(h[i]);
    }
}

rtcc_status parse_checkpoint(const void *file, size_t bytes, CkptView &v, std::string &err) {
    v = CkptView();
    if (!file) { err = "checkpoint pointer is NULL"; return RTCC_E_ARG; }
    const unsigned char *f = static_cast<const unsigned char *>(file);
    if (bytes < kCkptHeaderBytes) { err = "checkpoint shorter than its 128-byte header"; return RTCC_E_MALFORMED; }
    if (std::memcmp(f, kMagic, 8) != 0) { err = "not a weights checkpoint (magic)"; return RTCC_E_MALFORMED; }
    const uint32_t version = rd32(f + 8);
    if (version != kCkptVersion) {
        err = "checkpoint version " + std::to_string(version) + " (this library reads 1)";
        return RTCC_E_MALFORMED;
    }
    const uint32_t n_tensors = rd32(f + 12);
    std::string cfg_id;
    if (!nul_terminated(f + 16, 32, cfg_id)) { err = "config id is not NUL-terminated and zero-padded"; return RTCC_E_MALFORMED; }
    const uint64_t seed = rd64(f + 48);
    const uint64_t data_offset = rd64(f + 56);
    const uint64_t data_bytes = rd64(f + 64);
    for (size_t i = 104; i < kCkptHeaderBytes; ++i)
        if (f[i]) { err = "reserved header bytes are not zero"; return RTCC_E_MALFORMED; }
    if (n_tensors < 1 || n_tensors > 4096) { err = "tensor count out of range"; return RTCC_E_MALFORMED; }
    const uint64_t table_end = kCkptHeaderBytes + uint64_t(n_tensors) * kCkptEntryBytes;
    if (data_offset % 64 || data_offset < table_end || data_offset > bytes) {
        err = "data offset is not 64-aligned after the tensor table"; return RTCC_E_MALFORMED;
    }
    for (uint64_t i = table_end; i < data_offset; ++i)
        if (f[i]) { err = "padding before the data section is not zero"; return RTCC_E_MALFORMED; }
    if (data_bytes != bytes - data_offset) {
        err = "data section is " + std::to_string(bytes - data_offset) + " bytes, header says " +
              std::to_string(data_bytes);
        return RTCC_E_MALFORMED;
    }
    uint64_t next = 0;
    for (uint32_t t = 0; t < n_tensors; ++t) {
        const unsigned char *e = f + kCkptHeaderBytes + size_t(t) * kCkptEntryBytes;
        CkptTensor ct;
        const std::string where = "tensor " + std::to_string(t);
        if (!nul_terminated(e, 64, ct.name) || ct.name.empty()) { err = where + ": bad name"; return RTCC_E_MALFORMED; }
        if (rd32(e + 64) != 0) { err = where + " (" + ct.name + "): dtype is not float32"; return RTCC_E_MALFORMED; }
        ct.ndim = int(rd32(e + 68));
        if (ct.ndim < 1 || ct.ndim > 4) { err = where + " (" + ct.name + "): ndim out of [1, 4]"; return RTCC_E_MALFORMED; }
        uint64_t elems = 1;
        for (int d = 0; d < 4; ++d) {
            const int64_t s = int64_t(rd64(e + 72 + 8 * d));
            if (d < ct.ndim ? (s < 1 || s > (int64_t(1) << 31)) : s != 0) {
                err = where + " (" + ct.name + "): bad shape"; return RTCC_E_MALFORMED;
            }
            ct.shape[d] = s;
            if (d < ct.ndim) elems *= uint64_t(s);
            if (elems > (uint64_t(1) << 40)) { err = where + ": too large"; return RTCC_E_MALFORMED; }
        }
        ct.offset = rd64(e + 104);
        ct.nbytes = rd64(e + 112);
        for (int i = 120; i < 128; ++i)
            if (e[i]) { err = where + ": reserved bytes are not zero"; return RTCC_E_MALFORMED; }
        if (ct.nbytes != 4 * elems) { err = where + " (" + ct.name + "): nbytes != 4 x elements"; return RTCC_E_MALFORMED; }
        if (ct.offset != next) { err = where + " (" + ct.name + "): tensors are not back to back"; return RTCC_E_MALFORMED; }
        next += ct.nbytes;
        v.tensors.push_back(ct);
    }
    if (next != data_bytes) { err = "tensors do not cover the data section"; return RTCC_E_MALFORMED; }
    uint8_t digest[32];
    sha256(f + data_offset, size_t(data_bytes), digest);
    if (std::memcmp(digest, f + 72, 32) != 0) { err = "data section does not match its SHA-256"; return RTCC_E_MALFORMED; }

    std::memset(&v.info, 0, sizeof(v.info));
    std::memcpy(v.info.config_id, cfg_id.c_str(), cfg_id.size() + 1);
    v.info.seed = seed;
    v.info.version = int32_t(version);
    v.info.n_tensors = int32_t(n_tensors);
    v.info.data_bytes = data_bytes;
    std::memcpy(v.info.sha256, digest, 32);
    v.data = f + data_offset;
    return RTCC_OK;
}

std::vector<CkptTensor> expected_tensors(const Plan &p) {
    std::vector<CkptTensor> out;
    auto add = [&](const std::string &name, std::initializer_list<int64_t> shape) {
        CkptTensor t;
        t.name = name;
        t.ndim = int(shape.size());
        int d = 0;
        uint64_t elems = 1;
        for (int64_t s : shape) { t.shape[d++] = s; elems *= uint64_t(s); }
        t.nbytes = 4 * elems;
        out.push_back(t);
    };
    add("pfn_w", {4, p.c_pfn});
    add("pfn_b", {p.c_pfn});
    int l = 0, stage = -1;
    for (const ConvLayer &c : p.convs) {
        if (c.stage != stage) { stage = c.stage; l = 0; }
        const std::string base = "s" + std::to_string(c.stage) + "c" + std::to_string(l++);
        add(base + "_w", {3, 3, c.Ci, c.Co});
        add(base + "_b", {c.Co});
    }
    for (const UpLayer &u : p.ups) {
        const std::string base = "up" + std::to_string(u.stage);
        add(base + "_w", {u.u, u.u, u.Ci, u.Co});
        add(base + "_b", {u.Co});
    }
    add("head_w", {p.c_slot, 16});
    add("head_b", {16});
    uint64_t off = 0;
    for (CkptTensor &t : out) { t.offset = off; off += t.nbytes; }
    return out;
}

}  // namespace rtcc
