// Host-only helpers shared by the C ABI implementation and the packer.
#pragma once
#include <stdint.h>

#include "../../include/sph.h"

int sph_host_check_format(const sph_format* fmt);
int sph_host_check_shape(int64_t n, int64_t k);
int sph_host_layout(const sph_format* fmt, int64_t n, int64_t k, uint64_t off[8], uint64_t* total);
int sph_host_check_codes(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                         const uint16_t* dir_idx, const uint8_t* radius_code, const uint16_t* gmin,
                         const uint16_t* gstep, const uint16_t* codebook);
void sph_host_pack(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                   const uint16_t* dir_idx, const uint8_t* radius_code, const uint16_t* gmin,
                   const uint16_t* gstep, const uint16_t* codebook, const uint64_t off[8],
                   uint8_t* blob);
