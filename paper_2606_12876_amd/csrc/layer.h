// Internal definitions shared by the host library and the kernel launchers.
#pragma once
#include <cstddef>
#include <cstdint>

#include "../../include/aqmb.h"

namespace aqmb {

// Codes are stored per plane as [S slices][d_out rows][J groups]: a slice holds J
// consecutive groups of every row, so one 16-byte load brings the J codes of one
// row (J = 16 uint8 codes or 8 uint16 codes). Groups past d_in/g in the last slice
// are padding (code 0) and contribute nothing. Planes stay outermost: level k
// reads the first k * plane_bytes bytes only.
constexpr int kSliceBytes = 16;
constexpr size_t kZeroPageBytes = 1024;
constexpr size_t kAuxBytes = kZeroPageBytes + 256;

struct Layer {
  uint32_t magic;
  aqmb_desc d;
  int device;
  int n_cu;              // compute units of that device (persistent grids)
  int G;                 // groups per row = d_in / g
  int J;                 // groups per slice
  int S;                 // slices per row = ceil(G / J)
  size_t plane_bytes;    // S * d_out * 16
  int resident;          // planes 0..resident-1 are in memory (the others were never loaded or were dropped)
  unsigned char* codes;  // [resident][S][d_out][16 bytes]
  uint16_t* codebooks;   // [M][2^B][g] fp16
  uint16_t* scales;      // [d_out] fp16
  // 1 KiB of zeros that kernels read in place of inputs past their end (never written after
  // create), followed by one int that the code upload of create / load_planes uses to flag 4-bit
  // codes above 15. Compute calls never write layer memory, so they may overlap on any streams.
  unsigned char* aux;
  const void* zero_page() const { return aux; }
  int* upload_flag() const { return (int*)(aux + kZeroPageBytes); }
};

constexpr uint32_t kMagic = 0x41514D42u;  // "AQMB"

}  // namespace aqmb
