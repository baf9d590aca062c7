// Host round trip of the library's packer, built with AddressSanitizer and UndefinedBehavior-
// Sanitizer by tests/test_pack_roundtrip.py (test infrastructure, not part of the library).
//
// Reads logical codes from a binary file, validates and packs them with the library's host code
// (sph_host_layout, sph_host_check_codes, sph_host_pack) into a heap blob of exactly the size the
// layout reports, pre-filled with a canary byte, then reads every field back with a decoder of
// its own written from the layout description (csrc/sph_layout.h) and writes the decoded codes.
// It also checks, and reports through its exit status, that
//   - nothing was written between the end of one stream and the aligned start of the next,
//   - padded rows of the last 16-row tile decode to zero codes and zero group parameters,
//   - the lookup tables and the codebook copy follow from the codebook as the layout states.
//
// Input file: int32 vec_dim, dir_bits, radius_bits; int64 n, k; then signs [n][k/vec]
// (uint8, uint16 for vec 16), dir [n][k/vec] uint16, q [n][k/vec] uint8, gmin and gstep
// [n][k/128] uint16, codebook [2^D][vec] uint16. The output file holds the five code arrays
// in the same order and types.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../paper_2609_24875_amd/csrc/sph_host.h"
#include "../../paper_2609_24875_amd/csrc/sph_layout.h"

namespace {

constexpr uint8_t kCanary = 0xA5;

template <class T>
bool read_arr(FILE* f, std::vector<T>& v, size_t count) {
  v.resize(count);
  return count == 0 || fread(v.data(), sizeof(T), count, f) == count;
}

template <class T>
bool write_arr(FILE* f, const std::vector<T>& v) {
  return v.empty() || fwrite(v.data(), sizeof(T), v.size(), f) == v.size();
}

uint32_t ld32(const uint8_t* p) {
  uint32_t x;
  std::memcpy(&x, p, 4);
  return x;
}
uint16_t ld16(const uint8_t* p) {
  uint16_t x;
  std::memcpy(&x, p, 2);
  return x;
}

int fail(const char* what) {
  fprintf(stderr, "pack_roundtrip: %s\n", what);
  return 10;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) return fail("usage: pack_roundtrip <in> <out>");
  FILE* f = fopen(argv[1], "rb");
  if (!f) return fail("cannot open input");
  int32_t hdr[3];
  int64_t nk[2];
  if (fread(hdr, 4, 3, f) != 3 || fread(nk, 8, 2, f) != 2) return fail("short header");
  sph_format fmt{hdr[0], hdr[1], hdr[2], 128};
  const int64_t n = nk[0], k = nk[1];
  const int vec = fmt.vec_dim, D = fmt.dir_bits, V = fmt.radius_bits;
  if (sph_host_check_format(&fmt) != 0 || sph_host_check_shape(n, k) != 0) return fail("bad format or shape");
  const int64_t nvd = k / vec, ng = k / SPH_GROUP;
  std::vector<uint8_t> signs8;
  std::vector<uint16_t> signs16, dir, gmin, gstep, cb;
  std::vector<uint8_t> q;
  bool ok = vec == 16 ? read_arr(f, signs16, (size_t)(n * nvd)) : read_arr(f, signs8, (size_t)(n * nvd));
  ok = ok && read_arr(f, dir, (size_t)(n * nvd)) && read_arr(f, q, (size_t)(n * nvd));
  ok = ok && read_arr(f, gmin, (size_t)(n * ng)) && read_arr(f, gstep, (size_t)(n * ng));
  ok = ok && read_arr(f, cb, (size_t)vec << D);
  fclose(f);
  if (!ok) return fail("short input");
  const uint8_t* signs = vec == 16 ? (const uint8_t*)signs16.data() : signs8.data();

  uint64_t off[8], total = 0;
  if (sph_host_layout(&fmt, n, k, off, &total) != 0) return fail("layout");
  if (sph_host_check_codes(&fmt, n, k, signs, dir.data(), q.data(), gmin.data(), gstep.data(), cb.data()) != 0)
    return fail("codes rejected");
  uint8_t* blob = (uint8_t*)malloc(total);
  std::memset(blob, kCanary, total);
  sph_host_pack(&fmt, n, k, signs, dir.data(), q.data(), gmin.data(), gstep.data(), cb.data(), off, blob);

  const int kind = sph_kind_of_fmt(vec, D, V);
  const int64_t nt = (n + 15) / 16, nv = k / 8;
  // bytes each stream uses, from the layout description
  uint64_t used[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (sph_is_rowvec_kind(kind)) {
    used[SPH_OFF_A] = (uint64_t)(n * nvd) * (kind == SPH_KIND_V4 ? 1 : 4);
    used[SPH_OFF_B] = (uint64_t)(n * ng) * 4;
    used[SPH_OFF_PARAMS] = (uint64_t)(n * ng) * 4;
    used[SPH_OFF_TABLES] = sph_table_bytes(kind, D);
    used[SPH_OFF_CODEBOOK] = (uint64_t)vec * 2 << D;
  } else {
    used[SPH_OFF_A] = (uint64_t)(nt * nv) * 4 * sph_a_dwords(kind);
    used[SPH_OFF_B] = (uint64_t)(nt * nv) * 4 * sph_b_dwords(kind);
    used[SPH_OFF_PARAMS] = (uint64_t)(nt * ng) * 16 * 4;
    used[SPH_OFF_TABLES] = sph_table_bytes(kind, D);
    used[SPH_OFF_CODEBOOK] = (uint64_t)16 << D;
    used[SPH_OFF_C] = (uint64_t)(nt * nv) * 2 * sph_c_halves(kind);
  }
  // every byte outside the used extents keeps the canary
  std::vector<uint8_t> owned(total, 0);
  for (int s = 0; s < 6; ++s) {
    if (off[s] + used[s] > total) return fail("stream beyond the blob");
    for (uint64_t i = 0; i < used[s]; ++i) {
      if (owned[off[s] + i]) return fail("streams overlap");
      owned[off[s] + i] = 1;
    }
  }
  for (uint64_t i = 0; i < total; ++i)
    if (!owned[i] && blob[i] != kCanary) return fail("write outside every stream");

  std::vector<uint16_t> o_s16(vec == 16 ? n * nvd : 0), o_dir(n * nvd), o_gmin(n * ng), o_gstep(n * ng);
  std::vector<uint8_t> o_s8(vec == 16 ? 0 : n * nvd), o_q(n * nvd);
  const uint8_t* A = blob + off[SPH_OFF_A];
  const uint8_t* B = blob + off[SPH_OFF_B];
  const uint8_t* P = blob + off[SPH_OFF_PARAMS];
  const uint8_t* Cs = blob + off[SPH_OFF_C];
  const uint32_t zmask = (1u << D) - 1;

  if (sph_is_rowvec_kind(kind)) {
    for (int64_t row = 0; row < n; ++row)
      for (int64_t i = 0; i < nvd; ++i) {
        const int64_t x = row * nvd + i, g = i / (SPH_GROUP / vec), v = i % (SPH_GROUP / vec);
        const uint32_t b = ld32(B + (row * ng + g) * 4);
        if (kind == SPH_KIND_V4) {
          const uint8_t a = A[x];
          o_s8[x] = a & 15;
          o_dir[x] = (a >> 4) & 3;
          o_q[x] = (uint8_t)(((a >> 6) & 3) | (((b >> v) & 1) << 2));
        } else {
          const uint32_t a = ld32(A + x * 4);
          o_s16[x] = (uint16_t)(a & 0xFFFF);
          o_dir[x] = (uint16_t)((a >> 16) & 0x3FFF);
          o_q[x] = (uint8_t)((a >> 30) | (((b >> (4 * v)) & 15) << 2));
        }
      }
    for (int64_t i = 0; i < n * ng; ++i) {
      o_gmin[i] = ld16(P + i * 4);
      o_gstep[i] = ld16(P + i * 4 + 2);
    }
  } else {
    const int W = 8 + D;
    for (int64_t t = 0; t < nt; ++t)
      for (int64_t v = 0; v < nv; ++v) {
        const uint8_t* a = A + (t * nv + v) * 4 * sph_a_dwords(kind);
        const uint8_t* b = B + (t * nv + v) * 4 * sph_b_dwords(kind);
        for (int r = 0; r < 16; ++r) {
          uint32_t s = 0, z = 0, qq = 0;
          if (kind == SPH_KIND_W2) {
            const uint32_t w = ld32(a + 4 * (r / 2));
            const uint32_t fld = (r % 2 == 0) ? (w & ((1u << W) - 1)) : ((w >> W) & ((1u << W) - 1));
            s = (fld & 15) | (((fld >> (4 + D)) & 15) << 4);
            z = (fld >> 4) & zmask;
            qq = (r % 2 == 0) ? (w >> (2 * W)) : ((ld32(b) >> (4 * (r / 2))) & 15);
          } else if (kind == SPH_KIND_NIB16 || kind == SPH_KIND_NIB16Q8 || kind == SPH_KIND_NIB16Q2) {
            const uint32_t fld = ld16(a + 2 * r);
            s = (fld & 15) | (((fld >> (4 + D)) & 15) << 4);
            z = (fld >> 4) & zmask;
            if (kind == SPH_KIND_NIB16) qq = fld >> (8 + D);
            else if (kind == SPH_KIND_NIB16Q8) qq = b[r];
            else qq = (ld32(b) >> (2 * r)) & 3;
          } else {  // CB13, CB13Q4
            s = a[r];
            const uint32_t fld = ld16(b + 2 * r);
            z = fld & 0x1FFF;
            qq = fld >> 13;
            if (kind == SPH_KIND_CB13Q4) qq |= ((ld16(Cs + (t * nv + v) * 2) >> r) & 1u) << 3;
          }
          const int64_t row = t * 16 + r;
          if (row < n) {
            o_s8[row * nv + v] = (uint8_t)s;
            o_dir[row * nv + v] = (uint16_t)z;
            o_q[row * nv + v] = (uint8_t)qq;
          } else if (s || z || qq) {
            return fail("padded row with a non-zero code");
          }
        }
      }
    for (int64_t t = 0; t < nt; ++t)
      for (int64_t g = 0; g < ng; ++g)
        for (int r = 0; r < 16; ++r) {
          const uint32_t p = ld32(P + ((t * ng + g) * 16 + r) * 4);
          const int64_t row = t * 16 + r;
          if (row < n) {
            o_gmin[row * ng + g] = (uint16_t)(p & 0xFFFF);
            o_gstep[row * ng + g] = (uint16_t)(p >> 16);
          } else if (p) {
            return fail("padded row with non-zero group parameters");
          }
        }
  }

  // tables and codebook copy
  const uint8_t* T = blob + off[SPH_OFF_TABLES];
  const uint8_t* C = blob + off[SPH_OFF_CODEBOOK];
  const uint32_t entries = 1u << D;
  for (uint32_t i = 0; i < (uint32_t)vec * entries; ++i)
    if (ld16(C + 2 * i) != cb[i]) return fail("codebook copy");
  if (kind == SPH_KIND_V4) {
    for (uint32_t z = 0; z < entries; ++z)
      for (uint32_t s = 0; s < 16; ++s)
        for (int j = 0; j < 4; ++j)
          if (ld16(T + (((z << 4) | s) * 4 + j) * 2) != (uint16_t)(cb[z * 4 + j] ^ (((s >> j) & 1) ? 0x8000 : 0)))
            return fail("4-D table");
  } else if (sph_is_codebook_kind(kind)) {
    for (uint32_t i = 0; i < 8 * entries; ++i)
      if (ld16(T + 2 * i) != cb[i]) return fail("codebook table");
  } else if (!sph_is_rowvec_kind(kind)) {
    const uint8_t* Thi = T + (size_t)entries * 16 * 8;
    for (uint32_t z = 0; z < entries; ++z)
      for (uint32_t s = 0; s < 16; ++s)
        for (int j = 0; j < 4; ++j) {
          const uint16_t flip = ((s >> j) & 1) ? 0x8000 : 0;
          if (ld16(T + ((z * 16 + s) * 4 + j) * 2) != (uint16_t)(cb[z * 8 + j] ^ flip)) return fail("low table");
          if (ld16(Thi + ((s * entries + z) * 4 + j) * 2) != (uint16_t)(cb[z * 8 + 4 + j] ^ flip)) return fail("high table");
        }
  }
  free(blob);

  FILE* o = fopen(argv[2], "wb");
  if (!o) return fail("cannot open output");
  ok = vec == 16 ? write_arr(o, o_s16) : write_arr(o, o_s8);
  ok = ok && write_arr(o, o_dir) && write_arr(o, o_q) && write_arr(o, o_gmin) && write_arr(o, o_gstep);
  fclose(o);
  return ok ? 0 : fail("short output");
}
