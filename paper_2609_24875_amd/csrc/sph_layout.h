// Library-private device layout of a packed SPHQuant matrix (layout version 1).
//
// The logical representation is the one of Sec. 3.1 (Eq. 3-7): per 8-D vector a sign byte s,
// a D-bit direction index z and a V-bit radius level q; per 128-weight group of a row an fp16
// (offset, step) pair. This header fixes how those fields sit in device memory so that one lane
// can decode 16 rows of one vector position from 16-byte loads. It is included by the host
// packer and by the kernels; the layout is not part of the ABI.
//
// Rows are grouped into tiles of 16. Vector position v of tile t is one "record"; records are
// stored in order t * NV + v (NV = k/8) in up to three planar streams A, B, C. Within a record the
// 16 rows are r = 0..15 of the tile. Sign bits are split into the low nibble s_lo (elements
// 0..3) and the high nibble s_hi (elements 4..7).
//
//  kind W2       (D=6,V=4; D=6,V=3; D=7,V=2)
//                           A: 8 dwords, dword i = F(2i) | F(2i+1)<<W | q(2i)<<2W, W = 8+D,
//                             F(r) = s_lo | z<<4 | s_hi<<(4+D) (W bits; V <= 32-2W)
//                           B: 1 dword, bits [4i+3:4i] = q(2i+1)
//  kind NIB16    (D+V=8)    A: 8 dwords, 16-bit field per row (row r in dword r/2, half r%2):
//                             s_lo | z<<4 | s_hi<<(4+D) | q<<(8+D)
//                           B: none
//  kind NIB16Q8  (D=8,V=8)  A: 8 dwords, 16-bit field per row: s_lo | z<<4 | s_hi<<12
//                           B: 4 dwords, byte r = q(r)
//  kind NIB16Q2  (D=8,V=2)  A: as NIB16Q8
//                           B: 1 dword, bits [2r+1:2r] = q(r)
//  kind CB13     (D=13,V=3) A: 4 dwords, byte r = s(r)
//                           B: 8 dwords, 16-bit field per row: z | q<<13
//  kind CB13Q4   (D=13,V=4) A, B as CB13 with the low 3 bits of q in B
//                           C: one 16-bit word per record, bit r = bit 3 of q(r)
//
//  Row-planar kinds for 4-D and 16-D vectors (Tab. 7); no tiles, rows stored one after another:
//  kind V4  (vec 4, D=2, V=3)   A: one byte per vector [n][k/4]: s | z<<4 | (q & 3)<<6
//                               B: one dword per row and group [n][k/128]: bit v = q(v) >> 2
//                               table: 64 signed directions T[z<<4 | s] = 4 fp16 (sign-folded)
//  kind V16 (vec 16, D=14, V=6) A: one dword per vector [n][k/16]: s | z<<16 | (q & 3)<<30
//                               B: one dword per row and group: bits [4v+3:4v] = q(v) >> 2
//                               the codebook (2^14 x 16 fp16, 512 KiB) is read from memory
//  Group parameters of the row-planar kinds: half2 (offset, step) at [n][k/128].
//
// Nibble kinds (W2, NIB16*) look the signed direction up in two tables built from the codebook:
//   T_lo[z*16 + s_lo]   = 4 fp16: element j of c_z for j = 0..3, negated where bit j of s_lo is set
//   T_hi[s_hi*2^D + z]  = 4 fp16: element 4+j of c_z for j = 0..3, negated where bit j of s_hi is set
// so that the low table index is the field bits [D+3:0] and the high table index is the field
// bits [D+7:4]. The codebook kinds (CB13*) look up the unsigned entry c_z (16 bytes) and apply
// the signs with two 16-entry XOR-mask tables.
//
// Group parameters: half2 (x = offset, y = step) at ((t * NG + g) * 16 + r), NG = k/128.
// Padded rows (r >= n) carry zero codes and zero parameters, so they decode to zero.
#pragma once
#include <stdint.h>

#define SPH_LAYOUT_VERSION 1u
#define SPH_MAGIC 0x53504851u  // "SPHQ"
#define SPH_TILE_ROWS 16
#define SPH_VEC 8
#define SPH_GROUP 128
#define SPH_ALIGN 256

enum sph_kind {
  SPH_KIND_W2 = 0, SPH_KIND_NIB16 = 1, SPH_KIND_NIB16Q8 = 2, SPH_KIND_CB13 = 3, SPH_KIND_NIB16Q2 = 4,
  SPH_KIND_CB13Q4 = 5, SPH_KIND_V4 = 6, SPH_KIND_V16 = 7, SPH_KIND_NONE = -1
};

// Offsets inside the device blob (sph_weights.off[]).
enum sph_off {
  SPH_OFF_A = 0, SPH_OFF_B = 1, SPH_OFF_PARAMS = 2, SPH_OFF_TABLES = 3, SPH_OFF_CODEBOOK = 4, SPH_OFF_C = 5
};

static inline int sph_kind_of(int dir_bits, int radius_bits) {
  if ((dir_bits == 6 && (radius_bits == 4 || radius_bits == 3)) || (dir_bits == 7 && radius_bits == 2))
    return SPH_KIND_W2;
  if (dir_bits + radius_bits == 8 && dir_bits >= 4 && dir_bits <= 6 && radius_bits >= 2) return SPH_KIND_NIB16;
  if (dir_bits == 8 && radius_bits == 8) return SPH_KIND_NIB16Q8;
  if (dir_bits == 8 && radius_bits == 2) return SPH_KIND_NIB16Q2;
  if (dir_bits == 13 && radius_bits == 3) return SPH_KIND_CB13;
  if (dir_bits == 13 && radius_bits == 4) return SPH_KIND_CB13Q4;
  return SPH_KIND_NONE;
}

// Kind of a full format (vector size, D, V): 8-D formats as above; one 4-D and one 16-D format.
static inline int sph_kind_of_fmt(int vec_dim, int dir_bits, int radius_bits) {
  if (vec_dim == 8) return sph_kind_of(dir_bits, radius_bits);
  if (vec_dim == 4 && dir_bits == 2 && radius_bits == 3) return SPH_KIND_V4;
  if (vec_dim == 16 && dir_bits == 14 && radius_bits == 6) return SPH_KIND_V16;
  return SPH_KIND_NONE;
}

static inline bool sph_is_rowvec_kind(int kind) { return kind == SPH_KIND_V4 || kind == SPH_KIND_V16; }

// The codebook kinds keep c_z itself in LDS; the others keep the sign-folded nibble tables.
static inline bool sph_is_codebook_kind(int kind) { return kind == SPH_KIND_CB13 || kind == SPH_KIND_CB13Q4; }

// Dwords per record in streams A and B, 16-bit words per record in stream C.
static inline int sph_a_dwords(int kind) { return sph_is_codebook_kind(kind) ? 4 : 8; }
static inline int sph_b_dwords(int kind) {
  switch (kind) {
    case SPH_KIND_W2: return 1;
    case SPH_KIND_NIB16: return 0;
    case SPH_KIND_NIB16Q8: return 4;
    case SPH_KIND_NIB16Q2: return 1;
    case SPH_KIND_CB13: return 8;
    case SPH_KIND_CB13Q4: return 8;
    default: return 0;
  }
}
static inline int sph_c_halves(int kind) { return kind == SPH_KIND_CB13Q4 ? 1 : 0; }

// Bytes of the lookup tables kept in the blob: nibble kinds hold T_lo and T_hi (8 bytes per entry,
// 2^D * 16 entries each); codebook kinds hold the codebook as 16-byte entries.
static inline uint64_t sph_table_bytes(int kind, int dir_bits) {
  if (kind == SPH_KIND_V4) return 64 * 8;
  if (kind == SPH_KIND_V16) return 0;
  if (sph_is_codebook_kind(kind)) return (uint64_t)16 << dir_bits;
  return (uint64_t)2 * 8 * 16 << dir_bits;
}
