// Fused chain of small-block KS factors (paper Section 1 and Figure 1: a
// product of KS factors such as the butterfly factors of a fast transform;
// Appendix B.1, Table 5), shared by the kernel (ks_chain_fused.hip), the host
// planner (ks_host.cpp) and the host replay (ks_verify.hip).
//
// One workgroup owns a tile of kFusedCols batch columns and keeps the whole
// intermediate vector of each of its columns in LDS, in fp32, for the whole
// chain: X is read from HBM once, the factors are applied LDS -> LDS, and Y
// is written once.  Two forms: chains of small blocks (b, c <= 8) on the
// VALU, in radix passes (below, ks_chain_fused.hip), and chains whose blocks
// are all square with one b in {16, 32, 48, 64} (Monarch factors) on the fp32
// MFMAs (ks_chain_mfma.hip), one factor per pass, each block's outputs written
// over its own inputs (the index sets of a square block are the same rows)
// after the whole block is computed.
//
// The factors are applied in passes.  A radix pass applies m >= 1
// consecutive square factors with p x p blocks (applied order t = 0 .. m-1,
// factor t of pattern (a_t, p, p, d_t)) whose strides nest: d_{t+1} = p*d_t
// and a_t = a_{t+1}*p.  Then every block of every factor of the pass lies
// inside one of N / P groups of P = p^m rows,
//     rows(group) = { i*P*d_0 + j0 + d_0*r : r < P },  i < N/(P*d_0), j0 < d_0,
// and within a group factor t mixes the register digits r_t of
// r = sum_t r_t p^t: the p rows r + l*p^t (l < p, digit t of r zero) are the
// inputs l of block (i*P/(p^(t+1)) + r_hi, j0 + d_0*r_lo) of factor t, where
// r_lo < p^t and r_hi are the digits below and above t (Section 4.1 index
// sets: inputs i*c*d + l*d + j, outputs i*b*d + k*d + j, here with b = c = p).
// A work unit (group, 4 columns) loads its P rows into registers, applies the
// m factors there and stores them back in place: one LDS round trip for m
// factors.  Any other factor (b != c, or strides that do not nest) is a pass
// of its own: a unit reads the c input rows of one block and writes its b
// output rows, into the other LDS buffer when b != c.
//
// Factor values: each pass's values (its factors' packed blocks, one after
// the other) are fetched from global memory into registers one pass ahead
// (runs of 4 consecutive values per load when the buffers allow) and parked
// in an LDS copy as fp32 between passes.
//
// LDS layout: row r of the vector holds the tile's 16 columns at
// r * kFusedPitch floats (16 columns + 4 pad floats, so 16-byte accesses of
// consecutive rows spread over all banks); then the factor-value copy.  The
// MFMA form may take tiles of 32 columns (pitch 36) when they fit: every
// factor value it fetches then serves twice the columns.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

#include "ks_divide.h"

namespace ks {

constexpr int kFusedMaxFactors = 24;
constexpr int kFusedCols = 16;
constexpr int kFusedPitch = 20;                                  // floats per LDS row
constexpr int kFusedMaxBC = 8;                                   // largest b and c of a fused factor
constexpr int kFusedMaxLds = 160 * 1024;
constexpr int kFusedThreads = 512;                               // threads per workgroup
constexpr int kFusedKPerThread = 16;                             // factor values fetched per thread and pass
constexpr int kFusedKValues = kFusedThreads * kFusedKPerThread;  // largest value count of a pass (8192)
constexpr int kFusedMaxGroup = 8;                                // largest P = p^m of a radix pass
constexpr int kFusedMfmaMaxB = 64;                               // largest square block of the MFMA form

struct FusedChain {
  int nf;                   // factors, in product order (factor nf-1 is applied first)
  int batch;
  int layout;
  int width_in, width_out;  // a*c*d of factor nf-1, a*b*d of factor 0
  int inplace;              // every factor has b == c: one LDS buffer
  int buf_rows;             // rows of one LDS buffer (the widest vector)
  int kvec;                 // factor values fetched 4 at a time: every factor's count is a multiple
                            // of 4 and its values are aligned to 4 elements (set at launch)
  int mfma;                 // 1: square b x b blocks, one b in {16, 32, 48, 64}, on the fp32 MFMAs
                            // (ks_chain_mfma.hip), one factor per pass, in place, no factor-value copy
  int bfly;                 // L >= 2: the chain is the dyadic butterfly of size N = 2^L <= 1024
                            // (ks_chain_bfly.hip, two register passes); 0 otherwise
  int cols;                 // batch columns per workgroup tile: kFusedCols, or 2*kFusedCols for the
                            // MFMA form when the wider tile fits
  int pitch;                // floats per LDS row of the vector buffers (cols + 4)
  int a[kFusedMaxFactors], b[kFusedMaxFactors], c[kFusedMaxFactors], d[kFusedMaxFactors];
  uint32_t md[kFusedMaxFactors];  // multiply-shift constants of the division by d
  int sd[kFusedMaxFactors];
  const void* kv[kFusedMaxFactors];
  // passes, in application order; pass q applies factors pf0[q], pf0[q]-1, ...
  // (pm[q] of them); radix passes have pp[q] = p >= 2 and group size pP[q]
  int npass;
  int pf0[kFusedMaxFactors], pm[kFusedMaxFactors], pp[kFusedMaxFactors], pP[kFusedMaxFactors];
  int pk[kFusedMaxFactors];       // factor values of the pass (sum over its factors)
  int pcnt[kFusedMaxFactors];     // values of each factor of the pass (a*b*c*d, equal within a pass)
  uint32_t mgd[kFusedMaxFactors];  // multiply-shift division by the pass's d_0
  int sgd[kFusedMaxFactors];
  const void* x;
  void* y;
};

// Radix pass q: is it one (pp[q] >= 2)?  Its first factor's d is d_0.
__host__ __device__ __forceinline__ bool fused_is_radix(const FusedChain& fc, int q) { return fc.pp[q] >= 2; }

// Work units of radix pass q: (group, 16-byte piece), piece fastest.
__host__ __device__ __forceinline__ int fused_radix_units(const FusedChain& fc, int q) {
  const int f0 = fc.pf0[q];
  const int N = fc.a[f0] * fc.c[f0] * fc.d[f0];
  return N / fc.pP[q] * 4;
}
// Group g of radix pass q -> (i, j0): its rows are i*P*d_0 + j0 + d_0*r.
__host__ __device__ __forceinline__ void fused_radix_group(const FusedChain& fc, int q, int g, int* i, int* j0) {
  *i = (int)div_fast((uint32_t)g, fc.mgd[q], fc.sgd[q]);
  *j0 = g - *i * fc.d[fc.pf0[q]];
}
// Block index (i_t * d_t + j_t) of factor t of a radix pass with group size
// P and radix PR, acting on the register run r, r + p^t, ..., r + (p-1)*p^t
// (digit t of r zero) of group (i, j0); d_t = d_0 * p^t.
template <int P, int PR>
__host__ __device__ __forceinline__ int fused_radix_block(int i, int j0, int d0, int t, int r) {
  int st = 1;
  for (int u = 0; u < t; ++u) st *= PR;
  const int lo = r % st, hi = r / (st * PR);
  return (i * (P / (st * PR)) + hi) * (d0 * st) + j0 + d0 * lo;
}

// 16-byte pieces (4 columns each) of one LDS row handled by one work unit of
// a single-factor pass with blocks of at most m x m: two for m <= 2, one
// otherwise.
__host__ __device__ __forceinline__ int fused_pieces(int m) { return m <= 2 ? 2 : 1; }

// Work units of a single-factor pass over factor f: (block ij, group of
// pieces), group fastest.
__host__ __device__ __forceinline__ int fused_units(const FusedChain& fc, int f) {
  const int bc = fc.b[f] > fc.c[f] ? fc.b[f] : fc.c[f];
  return fc.a[f] * fc.d[f] * (4 / fused_pieces(bc));
}

// Block (i, j) and piece group g of work unit u of factor f (G = 4 / pieces
// groups per row); the kernel and the host replay share this decode.
__host__ __device__ __forceinline__ void fused_unit(const FusedChain& fc, int f, int G, int u, int* i, int* j,
                                                    int* g) {
  const int ij = u / G;
  *g = u - ij * G;
  *i = (int)div_fast((uint32_t)ij, fc.md[f], fc.sd[f]);
  *j = ij - *i * fc.d[f];
}
// LDS row of input l / output k of block (i, j) of factor f (Section 4.1
// index sets: columns i*c*d + l*d + j, rows i*b*d + k*d + j).
__host__ __device__ __forceinline__ int fused_in_row(const FusedChain& fc, int f, int i, int j, int l) {
  return i * fc.c[f] * fc.d[f] + l * fc.d[f] + j;
}
__host__ __device__ __forceinline__ int fused_out_row(const FusedChain& fc, int f, int i, int j, int k) {
  return i * fc.b[f] * fc.d[f] + k * fc.d[f] + j;
}

// Tile loads and stores, 16-byte form: unit u of a pass over the tile (of
// `cols` batch columns) covers E = 16 / sizeof(T) consecutive elements.
//  BSL: u -> (row n, column t0 = E * v), global element n*batch + col0 + t0,
//       LDS float n*kFusedPitch + t0 (+1 per element).
//  BSF: u -> (batch row t = u % 16, first element n0 = E * (u / 16)), global
//       element (col0 + t)*width + n0, LDS floats (n0 + e)*kFusedPitch + t.
__host__ __device__ __forceinline__ void fused_vec_unit(int layout, int E, int u, int* row, int* col,
                                                        int cols = kFusedCols) {
  if (layout == 1) {  // BSL
    const int pr = cols / E;
    *row = u / pr;
    *col = (u - *row * pr) * E;
  } else {
    // 16 batch rows x 4 consecutive pieces per 64 units (64-byte runs of each
    // batch row for 16-byte pieces), then the next 16 columns, then the next
    // 4 pieces; with 32 columns the width must be a multiple of 4 pieces
    const int h = (u >> 6) % (cols >> 4), kk = (u >> 6) / (cols >> 4);
    *col = (u & 15) + 16 * h;
    *row = (4 * kk + ((u >> 4) & 3)) * E;
  }
}

// Tile of workgroup `block` in a grid of `tiles`: workgroups are dispatched
// to the 8 XCDs round-robin (block % 8), so each XCD gets a contiguous range
// of tiles, taken in order; neighbouring tiles then share that XCD's L2.  In
// the batch-size-last layout a tile's row segments are 16 columns (32 or 64
// bytes), and the tiles sharing a 128-byte line run on one XCD instead of
// each fetching the whole line.  A bijection of [0, tiles) for any count.
__host__ __device__ __forceinline__ int fused_tile(int block, int tiles) {
  const int q = tiles >> 3, r = tiles & 7, x = block & 7, k = block >> 3;
  return x * q + (x < r ? x : r) + k;
}

// Butterfly form (ks_chain_bfly.hip): the chain is K_1 ... K_L with K_l of
// pattern (2^(l-1), 2, 2, 2^(L-l)), N = 2^L (paper Section 1 and Figure 1:
// the butterfly factors of a fast transform).  In application order factor
// s = L - l has d = 2^s, and its 2 x 2 block (i, j) mixes rows
// R = i*2d + j and R + d (Section 4.1 index sets with b = c = 2).  The L
// factors are split in two register passes: pass A applies s < LA = ceil(L/2)
// to groups of PA = 2^LA consecutive rows, pass B applies the rest to groups
// of PB = 2^(L-LA) rows j + PA*r.  A unit is (group, one batch column), so a
// pass has 16*N/P units; N <= 1024 keeps both at most 512 (one per thread).
__host__ __device__ __forceinline__ int bfly_la(int L) { return (L + 1) / 2; }
// Block of factor s (d = 2^s) that holds row R, and whether R is its second row.
__host__ __device__ __forceinline__ int bfly_block(int R, int s) {
  return (R >> (s + 1)) * (1 << s) + (R & ((1 << s) - 1));
}
// LDS row of vector row R (16 floats per row): rows of one pass-A group lie
// PA apart and rows of one pass-B group are consecutive across a wavefront,
// so XOR-ing the low two bits with (R >> LA) puts the four groups a wavefront
// touches in four different bank windows in both passes.
__host__ __device__ __forceinline__ int bfly_lds_row(int R, int la) { return R ^ ((R >> la) & 3); }
// LDS floats: the vector, N rows of 16 (the factor values stay in registers).
__host__ __device__ __forceinline__ int bfly_lds_floats(int N) { return N * 16; }

// LDS layout: the vector buffer(s), then the current pass's factor values.
__host__ __device__ __forceinline__ int fused_kbuf_offset(const FusedChain& fc) {
  return (fc.inplace ? 1 : 2) * fc.buf_rows * fc.pitch;  // floats
}
__host__ __device__ __forceinline__ int fused_lds_bytes(const FusedChain& fc) {
  if (fc.bfly) return bfly_lds_floats(fc.width_in) * 4;
  return (fused_kbuf_offset(fc) + (fc.mfma ? 0 : kFusedKValues)) * 4;
}

// MFMA form: every factor has b = c = 16*BT for one BT in 1 .. 4.  Work
// items of factor f are its a*d blocks, one wavefront each (all b output rows
// of the block for the tile's 16 columns); block index ij = i*d + j,
// wavefront w takes ij = w, w + W, ... (W = kFusedThreads / 64).
__host__ __device__ __forceinline__ int fused_mfma_bt(const FusedChain& fc) { return fc.b[0] / 16; }
// When the first factor applied has d = 1 its blocks are runs of B rows, and
// wavefront w loads the rows of its own blocks itself (no barrier first).
// Piece p (EP elements) of one block's B rows x NC columns of the tile, as
// (row offset r, column c).  BSL: EP consecutive columns of one row.  BSF: EP
// consecutive rows of one batch row; consecutive p run over 16 batch rows,
// then over the pieces of a row, so 64 lanes read 16 batch rows x 4 pieces.
__host__ __device__ __forceinline__ void fused_block_piece(int layout, int B, int NC, int EP, int p, int* r,
                                                           int* c) {
  if (layout == 1) {
    const int pr = NC / EP;
    *r = p / pr;
    *c = (p % pr) * EP;
  } else {
    const int kp = B / EP, m = p >> 4;
    *c = (p & 15) + 16 * ((m / kp) % (NC / 16));
    *r = (m % kp) * EP;
  }
}
__host__ __device__ __forceinline__ int fused_mfma_blocks(const FusedChain& fc, int f) { return fc.a[f] * fc.d[f]; }

}  // namespace ks
