// Kernel argument blocks and launch helpers shared by the WaveFilter
// kernels (device side) and the C-ABI (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wf {

constexpr int kBlock = 256;        // threads per workgroup, all kernels
constexpr int kMaxCoefTile = 64;   // coarse coefficients per skim tile
constexpr int kScanChunk = 128;    // pool tokens per scan workgroup
constexpr int kAttnChunk = 128;    // cache rows per attention workgroup
constexpr int kCoefPad = 4;        // fp32 pad per LDS coefficient row

enum CoefSource { kHaarSum = 0, kCascade = 1, kFromApprox = 2 };

struct DwtArgs {
  const void* K;       // [U][Ls][D]
  float* approx;       // [U][nJ][D]
  float* details;      // nullable, [U][L - nJ][D]
  long Ls;             // rows per unit in K (L: the transformed rows)
  int U, L, D, J, nJ;
  int cps;             // coefficients per stream
  int streams;         // streams per workgroup tile
  int ntiles;          // tiles per unit
  int boundary;        // 0 symmetric, 1 periodic
};

struct SkimTileArgs {
  const void* K;        // [U][L][D]      (Haar sum / cascade)
  const float* approx;  // [U][nJ][D]     (from approx)
  const void* Q;        // [U][B][D]
  float* logits;        // [U][B][nJ]
  float* stats;         // [U][ntiles][2][B]: row max, then row sum of exp
  const int32_t* parent;  // nullable: coefficient n is block 2 parent[n/2] + n%2
                          // of level J ([U][npar], ascending block ids at J + 1)
  int npar;
  long Ls;              // rows per unit in K (L: the filtered rows)
  int U, L, B, J, nJ;
  int cpt;              // coefficients per tile
  int ntiles;           // tiles per unit
  int boundary;
  float scale;
};

struct SkimSelectArgs {
  const float* logits;  // [U][B][nJ]
  const float* stats;   // [U][ntiles][2][B]
  float* W;             // [U][nJ] out
  int32_t* seg;         // [U][S] out (block ids), or [U][2S] tokens when pairs
  const int32_t* parent;  // nullable: candidate n is block 2 parent[n/2] + n%2
  int npar;
  int pairs;            // emit the two tokens of each kept 2-token block
  int U, B, nJ, ntiles, S;
};

struct ScanArgs {
  const void* Q;        // [U][B][D]
  const void* K;        // [U][L][D]
  const int32_t* seg;   // [U][S] (the regions; unused when the scan selects them)
  // the scan selects the regions itself (token-level path): W [U][nJ] of
  // the block weights kernel, the token skim's block rows [U][nJ][2][B]
  // (log-sum-exps of the selected blocks give the pool normalisers), and
  // seg_out [U][S] for the regions, written by the unit's first workgroup
  const float* W;
  const float* blocks;
  int32_t* seg_out;
  int nJ;
  int w_in_lds;         // W staged in LDS for the selection
  float* stats;         // [U][C][2][B]
  float* wpool;         // [U][P]  (weights mode)
  long Ls;              // rows per unit in K
  int U, L, B, J, S, P, C;
  int Cs;               // (max, sum) slices in `stats`: C, or 1 when precomputed
  int span;             // pool positions per workgroup (multiple of the chunk)
  int nbuf;             // LDS ring depth (bf16 path)
  int seg_cap;          // region ids staged per workgroup (bf16 path)
  float scale;
  // units per selection: the selecting scan of unit u reads W and writes
  // seg_out of selection u / share (seg_out by the group's first unit only)
  int share = 1;
};

struct ScanSelectArgs {
  const float* wpool;   // [U][P]
  const int32_t* seg;   // [U][S]
  int32_t* tok;         // [U][keff]
  int U, J, S, P, keff;
};

struct GatherArgs {
  const void* K;        // [U][L][D]
  const void* V;
  const int32_t* tok;   // [U][keff]
  const void* Kg;       // [U][G][D]
  const void* Vg;
  void* Ks;             // [U][keff + R + G][D]
  void* Vs;
  long Lf;              // first always-kept row: rows Lf .. L-1 follow tok
  int U, L, D, keff, R, G, elem;
};

struct AttnArgs {
  const void* Q;        // [U][B][D]
  const void* K;        // rows: [U][L][D] indexed by tok, or [U][nrows][D]
  const void* V;
  const int32_t* tok;   // nullable: rows are contiguous when null
  // the attention selects the tokens itself (token-level path): the top
  // nsel of the scan weights wpool [U][P] over the pool of the regions seg
  // [U][S] (2^J tokens each); tok_out [U][nsel] (nullable) receives them
  const float* wpool;
  const int32_t* seg;
  int32_t* tok_out;
  int P, S, J;
  int w_in_lds;         // wpool staged in LDS for the selection
  const void* Kg;       // [U][G][D] tail (indexed mode only)
  const void* Vg;
  float* part;          // [U][NS][B][D] unnormalised partial outputs
  float* pstat;         // [U][NS][2][B] partial row max, row sum
  void* O;              // [U][B][D]
  long Lf;              // indexed mode: rows Lf .. Lf + R - 1 of K/V follow tok
  int R;
  int U, L, B, nsel, G, nrows, NS;
  int rps;              // cache rows per split (multiple of the chunk)
  int nbuf;             // LDS ring depth (bf16 path)
  float scale;
  // units per selection: the selecting attention of unit u reads wpool and
  // seg of selection u / share (tok_out by the group's first unit only)
  int share = 1;
};

constexpr int kFastMaxQBlocks = 4;  // query rows <= 64 on the token-level skim

struct TokenSkimArgs {
  const void* K;        // [U][L][D] bf16
  const void* Q;        // [U][B][D] bf16
  float* blocks;        // [U][nJ][2][B]: coarse logits, then log-sum-exps of
                        // the block's token logits; without the log-sum-exps
                        // [U][B][nJ] coarse logits
  float* wstats;        // [U][R][2][B] coarse-logit max and sum of exp per range
  long Ls;              // rows per unit in K (L: the filtered rows)
  int U, L, B, nJ, R;
  int span;             // tokens per range (multiple of the chunk)
  int nbuf;             // LDS ring depth
  float scale;          // logit scale
  float norm;           // 2^{-J/2}
  // nullable: the rows are the gathered sequence of the kept blocks
  // parent [U][npar] of 2^pshift tokens each (a refinement scale of the
  // recursion); L then counts gathered rows
  const int32_t* parent;
  int npar, pshift;
  int par_cap;          // parent ids staged in LDS per range
};

// Daubechies-2 at J = 6 for the token-level skim: the level-6 low-pass filter
// f_6 (190 taps, zero-padded) and the three symmetric-end filters E_0 | E_1
// | E_2 (64, 128 and 192 taps).
struct Db2TokenTaps {
  float band[3 << 6];
  float edge[6 << 6];
};

// out [groups][n] = the sum over h < H of in [groups H + h][n], h in order
struct HeadSumArgs {
  const float* in;
  float* out;
  long n;
  int H, groups;
};

struct BlockWeightsArgs {
  const float* blocks;  // [U][nJ][2][B] block rows of the token skim
  const float* wstats;  // [U][R][2][B]
  float* W;             // [U][nJ] out
  int U, B, nJ, R;
  int WPU;              // workgroups (block slices) per unit
};

}  // namespace wf
