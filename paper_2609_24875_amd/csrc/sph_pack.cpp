#include <stdint.h>
// Host side of the library: argument validation and packing of logical SPHQuant codes
// (Sec. 3.1, Eq. 3-7) into the device layout described in sph_layout.h. Pure C++: no HIP
// headers, so it also builds and runs with g++ on a machine without a GPU.
#include <cmath>
#include <cstring>
#include <vector>

#include "sph_layout.h"
#include "sph_host.h"

static inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

static bool f16_finite(uint16_t b) { return ((b >> 10) & 0x1F) != 0x1F; }
static bool f16_sign(uint16_t b) { return (b >> 15) != 0; }

int sph_host_check_format(const sph_format* fmt) {
  if (!fmt) return SPH_ERR_NULL;
  if (fmt->group_size != SPH_GROUP) return SPH_ERR_UNSUPPORTED_FORMAT;
  if (sph_kind_of_fmt(fmt->vec_dim, fmt->dir_bits, fmt->radius_bits) == SPH_KIND_NONE) return SPH_ERR_UNSUPPORTED_FORMAT;
  return SPH_OK;
}

int sph_host_check_shape(int64_t n, int64_t k) {
  if (n < 1 || n > (int64_t(1) << 24)) return SPH_ERR_SHAPE;
  if (k < SPH_GROUP || k % SPH_GROUP != 0 || k > (int64_t(1) << 20)) return SPH_ERR_SHAPE;
  // records (16-row tiles x vector positions) are counted in 32 bits by the kernels' work plans
  if ((n + SPH_TILE_ROWS - 1) / SPH_TILE_ROWS * (k / SPH_VEC) > INT32_MAX) return SPH_ERR_SHAPE;
  return SPH_OK;
}

int sph_host_layout(const sph_format* fmt, int64_t n, int64_t k, uint64_t off[8], uint64_t* total) {
  int st = sph_host_check_format(fmt);
  if (st) return st;
  st = sph_host_check_shape(n, k);
  if (st) return st;
  const int kind = sph_kind_of_fmt(fmt->vec_dim, fmt->dir_bits, fmt->radius_bits);
  const uint64_t nt = (uint64_t)((n + SPH_TILE_ROWS - 1) / SPH_TILE_ROWS);
  const uint64_t nv = (uint64_t)(k / SPH_VEC), ng = (uint64_t)(k / SPH_GROUP);
  uint64_t p = 0;
  for (int i = 0; i < 8; ++i) off[i] = 0;
  if (sph_is_rowvec_kind(kind)) {
    const uint64_t nvd = (uint64_t)(k / fmt->vec_dim), fb = kind == SPH_KIND_V4 ? 1 : 4;
    off[SPH_OFF_A] = p;
    p = align_up(p + (uint64_t)n * nvd * fb, SPH_ALIGN);
    off[SPH_OFF_B] = p;
    p = align_up(p + (uint64_t)n * ng * 4, SPH_ALIGN);
    off[SPH_OFF_PARAMS] = p;
    p = align_up(p + (uint64_t)n * ng * 4, SPH_ALIGN);
    off[SPH_OFF_TABLES] = p;
    p = align_up(p + sph_table_bytes(kind, fmt->dir_bits), SPH_ALIGN);
    off[SPH_OFF_CODEBOOK] = p;
    p = align_up(p + ((uint64_t)fmt->vec_dim * 2 << fmt->dir_bits), SPH_ALIGN);
    off[SPH_OFF_C] = p;
    *total = p;
    return SPH_OK;
  }
  off[SPH_OFF_A] = p;
  p = align_up(p + nt * nv * 4 * sph_a_dwords(kind), SPH_ALIGN);
  off[SPH_OFF_B] = p;
  p = align_up(p + nt * nv * 4 * sph_b_dwords(kind), SPH_ALIGN);
  off[SPH_OFF_PARAMS] = p;
  p = align_up(p + nt * ng * SPH_TILE_ROWS * 4, SPH_ALIGN);
  off[SPH_OFF_TABLES] = p;
  p = align_up(p + sph_table_bytes(kind, fmt->dir_bits), SPH_ALIGN);
  off[SPH_OFF_CODEBOOK] = p;
  p = align_up(p + ((uint64_t)16 << fmt->dir_bits), SPH_ALIGN);
  off[SPH_OFF_C] = p;
  p = align_up(p + nt * nv * 2 * sph_c_halves(kind), SPH_ALIGN);
  *total = p;
  return SPH_OK;
}

int sph_host_check_codes(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                         const uint16_t* dir_idx, const uint8_t* radius_code, const uint16_t* gmin,
                         const uint16_t* gstep, const uint16_t* codebook) {
  if (!signs || !dir_idx || !radius_code || !gmin || !gstep || !codebook) return SPH_ERR_NULL;
  const int vec = fmt->vec_dim;
  const int64_t nvec = n * (k / vec), ngrp = n * (k / SPH_GROUP);
  const uint32_t dmax = 1u << fmt->dir_bits, qmax = 1u << fmt->radius_bits;
  for (int64_t i = 0; i < nvec; ++i)
    if (dir_idx[i] >= dmax || radius_code[i] >= qmax) return SPH_ERR_CODE_RANGE;
  if (vec == 4)
    for (int64_t i = 0; i < nvec; ++i)
      if (signs[i] >= 16) return SPH_ERR_CODE_RANGE;
  for (int64_t i = 0; i < ngrp; ++i) {
    if (!f16_finite(gmin[i])) return SPH_ERR_BAD_VALUE;
    if (!f16_finite(gstep[i]) || f16_sign(gstep[i])) return SPH_ERR_BAD_VALUE;
  }
  // Codebook entries are coordinates of non-negative unit directions (Sec. 3.1), so they lie in
  // [0, 1] up to rounding; entries above 2 (fp16 0x4000) are rejected. The bound keeps a level
  // times an entry (at most 255 * 2) far inside the fp16 range of the matrix-core operands.
  for (int64_t i = 0; i < ((int64_t)vec << fmt->dir_bits); ++i)
    if (!f16_finite(codebook[i]) || f16_sign(codebook[i]) || codebook[i] > 0x4000) return SPH_ERR_BAD_VALUE;
  return SPH_OK;
}

// Row-planar packing of the 4-D and 16-D formats (see sph_layout.h). For 16-D vectors the sign
// array holds one little-endian uint16 per vector.
static void pack_rowvec(const sph_format* fmt, int kind, int64_t n, int64_t k, const uint8_t* signs,
                        const uint16_t* dir_idx, const uint8_t* radius_code, const uint16_t* gmin,
                        const uint16_t* gstep, const uint16_t* codebook, const uint64_t off[8], uint8_t* blob) {
  const int vec = fmt->vec_dim;
  const int64_t nvd = k / vec, ng = k / SPH_GROUP, vpg = SPH_GROUP / vec;
  uint32_t* B = (uint32_t*)(blob + off[SPH_OFF_B]);
  uint32_t* P = (uint32_t*)(blob + off[SPH_OFF_PARAMS]);
  const uint16_t* s16 = (const uint16_t*)signs;
  for (int64_t row = 0; row < n; ++row) {
    for (int64_t g = 0; g < ng; ++g) {
      uint32_t b = 0;
      for (int64_t v = 0; v < vpg; ++v) {
        const int64_t i = row * nvd + g * vpg + v;
        const uint32_t q = radius_code[i], z = dir_idx[i];
        if (kind == SPH_KIND_V4) {
          blob[off[SPH_OFF_A] + i] = (uint8_t)((signs[i] & 15) | (z << 4) | ((q & 3) << 6));
          b |= ((q >> 2) & 1) << v;
        } else {
          ((uint32_t*)(blob + off[SPH_OFF_A]))[i] = (uint32_t)s16[i] | (z << 16) | ((q & 3) << 30);
          b |= ((q >> 2) & 15) << (4 * v);
        }
      }
      B[row * ng + g] = b;
      P[row * ng + g] = (uint32_t)gmin[row * ng + g] | ((uint32_t)gstep[row * ng + g] << 16);
    }
  }
  const uint32_t entries = 1u << fmt->dir_bits;
  if (kind == SPH_KIND_V4) {
    uint16_t* T = (uint16_t*)(blob + off[SPH_OFF_TABLES]);
    for (uint32_t z = 0; z < entries; ++z)
      for (uint32_t s = 0; s < 16; ++s)
        for (int j = 0; j < 4; ++j) T[((z << 4) | s) * 4 + j] = codebook[z * 4 + j] ^ (((s >> j) & 1) ? 0x8000 : 0);
  }
  std::memcpy(blob + off[SPH_OFF_CODEBOOK], codebook, sizeof(uint16_t) * vec * entries);
}

// One row's code, or zeros for a padding row.
struct Code {
  uint32_t s, z, q;
};

void sph_host_pack(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                   const uint16_t* dir_idx, const uint8_t* radius_code, const uint16_t* gmin,
                   const uint16_t* gstep, const uint16_t* codebook, const uint64_t off[8],
                   uint8_t* blob) {
  const int kind = sph_kind_of_fmt(fmt->vec_dim, fmt->dir_bits, fmt->radius_bits);
  if (sph_is_rowvec_kind(kind)) {
    pack_rowvec(fmt, kind, n, k, signs, dir_idx, radius_code, gmin, gstep, codebook, off, blob);
    return;
  }
  const int D = fmt->dir_bits;
  const int64_t nt = (n + SPH_TILE_ROWS - 1) / SPH_TILE_ROWS, nv = k / SPH_VEC, ng = k / SPH_GROUP;
  const int adw = sph_a_dwords(kind), bdw = sph_b_dwords(kind);
  uint32_t* A = (uint32_t*)(blob + off[SPH_OFF_A]);
  uint32_t* B = (uint32_t*)(blob + off[SPH_OFF_B]);
  uint32_t* P = (uint32_t*)(blob + off[SPH_OFF_PARAMS]);
  uint16_t* Cs = (uint16_t*)(blob + off[SPH_OFF_C]);
  const int W = 8 + D;                       // field width of kind W2

  for (int64_t t = 0; t < nt; ++t) {
    for (int64_t v = 0; v < nv; ++v) {
      Code c[SPH_TILE_ROWS];
      for (int r = 0; r < SPH_TILE_ROWS; ++r) {
        const int64_t row = t * SPH_TILE_ROWS + r;
        if (row < n) {
          const int64_t i = row * nv + v;
          c[r] = {signs[i], dir_idx[i], radius_code[i]};
        } else {
          c[r] = {0, 0, 0};
        }
      }
      uint32_t* a = A + (t * nv + v) * adw;
      uint32_t* b = B + (t * nv + v) * bdw;
      for (int i = 0; i < adw; ++i) a[i] = 0;
      for (int i = 0; i < bdw; ++i) b[i] = 0;
      switch (kind) {
        case SPH_KIND_W2:
          for (int i = 0; i < 8; ++i) {
            const Code& e = c[2 * i];
            const Code& o = c[2 * i + 1];
            const uint32_t fe = (e.s & 15) | (e.z << 4) | ((e.s >> 4) << (4 + D));
            const uint32_t fo = (o.s & 15) | (o.z << 4) | ((o.s >> 4) << (4 + D));
            a[i] = fe | (fo << W) | (e.q << (2 * W));
            b[0] |= o.q << (4 * i);
          }
          break;
        case SPH_KIND_NIB16:
          for (int r = 0; r < 16; ++r) {
            const uint32_t f = (c[r].s & 15) | (c[r].z << 4) | ((c[r].s >> 4) << (4 + D)) | (c[r].q << (8 + D));
            a[r / 2] |= (f & 0xFFFF) << (16 * (r % 2));
          }
          break;
        case SPH_KIND_NIB16Q8:
          for (int r = 0; r < 16; ++r) {
            const uint32_t f = (c[r].s & 15) | (c[r].z << 4) | ((c[r].s >> 4) << 12);
            a[r / 2] |= (f & 0xFFFF) << (16 * (r % 2));
            b[r / 4] |= (c[r].q & 0xFF) << (8 * (r % 4));
          }
          break;
        case SPH_KIND_NIB16Q2:
          for (int r = 0; r < 16; ++r) {
            const uint32_t f = (c[r].s & 15) | (c[r].z << 4) | ((c[r].s >> 4) << 12);
            a[r / 2] |= (f & 0xFFFF) << (16 * (r % 2));
            b[0] |= (c[r].q & 3) << (2 * r);
          }
          break;
        case SPH_KIND_CB13:
        case SPH_KIND_CB13Q4: {
          uint32_t hi = 0;
          for (int r = 0; r < 16; ++r) {
            a[r / 4] |= (c[r].s & 0xFF) << (8 * (r % 4));
            b[r / 2] |= ((c[r].z & 0x1FFF) | ((c[r].q & 7) << 13)) << (16 * (r % 2));
            hi |= ((c[r].q >> 3) & 1) << r;
          }
          if (kind == SPH_KIND_CB13Q4) Cs[t * nv + v] = (uint16_t)hi;
          break;
        }
      }
    }
    for (int64_t g = 0; g < ng; ++g)
      for (int r = 0; r < SPH_TILE_ROWS; ++r) {
        const int64_t row = t * SPH_TILE_ROWS + r;
        uint32_t pr = 0;
        if (row < n) pr = (uint32_t)gmin[row * ng + g] | ((uint32_t)gstep[row * ng + g] << 16);
        P[(t * ng + g) * SPH_TILE_ROWS + r] = pr;
      }
  }

  // Lookup tables derived from the codebook.
  uint16_t* T = (uint16_t*)(blob + off[SPH_OFF_TABLES]);
  const uint32_t entries = 1u << D;
  if (sph_is_codebook_kind(kind)) {
    for (uint32_t z = 0; z < entries; ++z)
      for (int j = 0; j < 8; ++j) T[z * 8 + j] = codebook[z * 8 + j];
  } else {
    uint16_t* Tlo = T;
    uint16_t* Thi = T + (size_t)entries * 16 * 4;
    for (uint32_t z = 0; z < entries; ++z)
      for (uint32_t s = 0; s < 16; ++s)
        for (int j = 0; j < 4; ++j) {
          const uint16_t flip = ((s >> j) & 1) ? 0x8000 : 0;
          Tlo[(z * 16 + s) * 4 + j] = codebook[z * 8 + j] ^ flip;
          Thi[(s * entries + z) * 4 + j] = codebook[z * 8 + 4 + j] ^ flip;
        }
  }
  uint16_t* C = (uint16_t*)(blob + off[SPH_OFF_CODEBOOK]);
  std::memcpy(C, codebook, sizeof(uint16_t) * 8 * entries);
}
