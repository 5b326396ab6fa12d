// Host-side plans and launchers of the WaveFilter kernels (used by the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "wavefilter.h"

namespace wf {

// Scores up to this many floats are staged in LDS by the select kernels.
constexpr int kSelectLdsFloats = 16384;
// region ids a select kernel keeps in LDS (more are read from global memory)
constexpr int kSelectLdsSegs = 8192;

struct DwtPlan {
  int streams;  // streams per workgroup
  int cps;      // coefficients per stream
  int ntiles;   // workgroups per unit
};

struct SkimPlan {
  int source;        // CoefSource
  int cpt;           // coefficients per tile
  int ntiles;        // tiles per unit
  size_t lds_bytes;  // dynamic LDS of the tile kernel
};

struct ScanPlan {
  int chunks;        // workgroups per unit
  int span;          // pool positions per workgroup
  int nbuf;          // LDS ring depth (bf16)
  int seg_cap;       // region ids staged per workgroup (bf16)
  size_t lds_bytes;  // dynamic LDS of the chunk kernels
};

struct AttnPlan {
  int splits;        // workgroups (row splits) per unit
  int rps;           // cache rows per split
  int nbuf;          // LDS ring depth (bf16)
  size_t lds_bytes;
};

struct FastPlan {
  int R;             // ranges (workgroups) per unit
  int span;          // tokens per range
  int nbuf;          // LDS ring depth
  int par_cap;       // parent ids staged per range (gathered rows), else 0
  size_t lds_bytes;
  bool held;         // block results kept in registers until the range's keys are read
};

// Workspace extents of the multi-scale recursion (maxima over its scales).
struct RecPlan {
  long max_n = 0;      // candidates of the widest scale
  int max_tiles = 0;   // coefficient tiles of the widest scale
  long max_keep = 0;   // kept blocks of the widest selection
};

float effective_scale(const wf_params& p);

// Filtered prompt rows: ctx_len rounded down to a multiple of 2^levels; the
// remaining ctx_len - filtered_len rows are always kept after the selection.
inline long filtered_len(const wf_params& p) {
  return ((long)p.ctx_len >> p.levels) << p.levels;
}
inline long remainder_len(const wf_params& p) { return (long)p.ctx_len - filtered_len(p); }
int device_cu_count();

DwtPlan plan_dwt(const wf_params& p);
SkimPlan plan_skim(const wf_params& p, bool fused);
// select: the scan workgroups take the top-S regions themselves (all S
// region ids in LDS)
ScanPlan plan_scan(const wf_params& p, bool select = false);
AttnPlan plan_attn(const wf_params& p, long nrows);

// The fused path streams the keys once with token-level scores when the keys
// are bf16, the wavelet is Haar with 3..5 levels and the query block has at
// most 64 rows; the scan then needs only its weights pass.
bool fast_path(const wf_params& p);
// The Daubechies-2 form of that path (J = 6, at least 4 coefficients).
bool db2_token_path(const wf_params& p);
// f_J (J <= 6) and the symmetric-end filters, computed in double.
void db2_token_taps(int J, Db2TokenTaps* out);
FastPlan plan_fast(const wf_params& p);
hipError_t launch_token_skim(const wf_params& p, const void* Q, const void* K,
                             float* blocks, float* wstats, hipStream_t s);
// W (eq. 8) of every coarse block from the token skim's block rows, by
// weights_slices(p) workgroups per unit.
int weights_slices(const wf_params& p);
hipError_t launch_block_weights(const wf_params& p, const float* blocks,
                                const float* wstats, float* W, hipStream_t s);

hipError_t launch_dwt(const wf_params& p, const void* K, float* approx,
                      float* details, hipStream_t s);
hipError_t launch_skim_tiles(const wf_params& p, bool fused, const void* Q,
                             const void* K, const float* approx, float* logits,
                             float* stats, hipStream_t s);
// One scale b of the multi-scale recursion (Haar).  Tiles: the coarse
// logits of its n candidates (all 2^b-blocks when parent is null, else the
// two halves of each block in parent [U][npar]).  Select: the eq. 8 weights
// and the top `keep`, written to out as block ids (b > 1) or as the two
// tokens of each kept block (b = 1).
RecPlan plan_recursion(const wf_params& p, const int32_t* counts);
hipError_t launch_rec_tiles(const wf_params& p, int b, long n, const int32_t* parent,
                            int npar, const void* Q, const void* K, float* logits,
                            float* stats, hipStream_t s);
hipError_t launch_rec_select(const wf_params& p, int b, long n, int keep,
                             const int32_t* parent, int npar, const float* logits,
                             const float* stats, float* W, int32_t* out, hipStream_t s);
// A scale b <= 5 of the recursion from token logits (bf16 keys, Haar, at
// most 64 query rows): over all filtered keys when parent is null (b =
// levels), else over the gathered kept blocks parent [U][npar] of 2^(b+1)
// tokens.  Writes the same n coarse logits per query row as the tiles
// ([U][B][n]) and one (max, sum) slice per range; the select then merges
// plan_rec_token(..).R slices.
bool rec_token_path(const wf_params& p);
FastPlan plan_rec_token(const wf_params& p, int b, long rows, bool gather);
hipError_t launch_rec_token_skim(const wf_params& p, int b, long n, const int32_t* parent,
                                 int npar, const void* Q, const void* K, float* logits,
                                 float* stats, hipStream_t s);
hipError_t launch_rec_select_slices(const wf_params& p, int b, long n, int keep,
                                    const int32_t* parent, int npar, int nslices,
                                    const float* logits, const float* stats, float* W,
                                    int32_t* out, hipStream_t s);
hipError_t launch_skim_select(const wf_params& p, int ntiles,
                              const float* logits, const float* stats,
                              float* W, int32_t* seg, hipStream_t s);
// W [U][nJ] of the coarse logits [U][B][nJ] and their tiles' (max, sum)
// pairs, spread over enough workgroups per unit to fill the chip (no
// selection); nJ must be a multiple of 4.
hipError_t launch_skim_weights(const wf_params& p, int ntiles, const float* logits,
                               const float* stats, float* W, hipStream_t s);
// stat_slices: 0 when `stats` holds one (max, sum) slice per scan workgroup
// (written by the stats pass), 1 when it holds the pool's final pair.
// share: units per selection (seg indexed by u / share).
hipError_t launch_scan_chunks(const wf_params& p, int weights, const void* Q,
                              const void* K, const int32_t* seg, float* stats,
                              float* wpool, hipStream_t s, int stat_slices = 0,
                              int share = 1);
// Token-level path: the weights pass that first takes the unit's top-S
// regions of W itself (seg_out [U][S] receives them) and forms the pool
// normalisers from the selected blocks' log-sum-exps (blocks [U][nJ][2][B]).
// share: units per selection (W and seg_out indexed by u / share; 1 = per
// unit).
hipError_t launch_scan_select_weights(const wf_params& p, const void* Q, const void* K,
                                      const float* W, const float* blocks, int32_t* seg_out,
                                      float* wpool, hipStream_t s, int share = 1);
// Whether the scan's workgroups can take the top-S regions themselves (bf16,
// at most 64 query rows, the region ids and the selection fit in LDS).
bool scan_can_select(const wf_params& p);
// The statistics pass that first takes the unit's top-S regions of W itself
// (seg_out [U][S] receives them, for the weights pass that follows) and
// writes one (max, sum) slice per workgroup into stats.
hipError_t launch_scan_select_stats(const wf_params& p, const void* Q, const void* K,
                                    const float* W, int32_t* seg_out, float* stats,
                                    hipStream_t s);
hipError_t launch_scan_select(const wf_params& p, const float* wpool,
                              const int32_t* seg, int32_t* tok,
                              hipStream_t s);
hipError_t launch_gather(const wf_params& p, const void* K, const void* V,
                         const int32_t* tok, const void* Kg, const void* Vg,
                         void* Ks, void* Vs, hipStream_t s);
// share: units per selection (tok indexed by u / share).
hipError_t launch_attn(const wf_params& p, const void* Q, const void* K,
                       const void* V, const int32_t* tok, int nsel,
                       const void* Kg, const void* Vg, int G, long nrows,
                       float* part, float* pstat, hipStream_t s, int share = 1);
// The top-S regions (eq. 9) of given weights W [groups][L >> J], one
// workgroup per group, into seg [groups][S].
hipError_t launch_select_w(const wf_params& p, long groups, const float* W, int32_t* seg,
                           hipStream_t s);
// Token-level path: the attention that first takes the unit's top-k_eff
// tokens of the scan weights wpool [U][S 2^J] itself (the pool of the
// regions seg [U][S]); tok_out [U][k_eff] (nullable) receives them.
bool attn_can_select(const wf_params& p, long nrows);
// share: units per selection (wpool, seg and tok_out indexed by u / share).
hipError_t launch_attn_select(const wf_params& p, const void* Q, const void* K, const void* V,
                              const float* wpool, const int32_t* seg, int32_t* tok_out,
                              const void* Kg, const void* Vg, long nrows, float* part,
                              float* pstat, hipStream_t s, int share = 1);
// out [groups][n] = sum over h < H of in [groups H + h][n], in order of h
// (the selection weights of a sequence's heads added up).
hipError_t launch_head_sum(const float* in, float* out, long n, int H, int groups,
                           hipStream_t s);
// Loads the code object of one translation unit onto the current device
// (each .hip file is its own code object; asking for a kernel's attributes
// loads it).
hipError_t load_fast_kernels();
hipError_t load_scan_kernels();
hipError_t load_attn_kernels();
hipError_t load_skim_kernels();
hipError_t launch_attn_combine(const wf_params& p, long nrows,
                               const float* part, const float* pstat, void* O,
                               hipStream_t s);

}  // namespace wf
