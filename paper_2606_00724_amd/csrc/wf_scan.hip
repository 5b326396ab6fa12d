// Scan: the skim's regions mapped to token indices (eq. 10) and scored at
// token resolution with the same perception-weight procedure (eqs. 7-8 over
// the pool only, Section 3.2), then the top-k tokens (eq. 9) -> mu^0.
//
// The pool of a unit is S runs of 2^J consecutive rows.  It is split into
// chunks of kScanChunk pool positions, one workgroup each.  The softmax over
// the pool needs every chunk's row maximum and normaliser before any weight
// can be formed, so the scan runs as two passes over the chunks:
//   pass 1 (stats):   logits of the chunk on MFMA, per-row max and
//                     sum of exp -> workspace;
//   pass 2 (weights): merge the unit's row statistics, recompute the same
//                     logits (bit-identical: same code and operands), and
//                     W'_p = sum_q exp(s_qp - M_q) / Z_q for the chunk.
// A per-unit select kernel then takes the top-k of W' (ties to the lower
// pool position, which is the lower token index because the regions are
// ascending) and emits token indices in ascending order.
#include "wf_device.hpp"
#include "wf_kernels.hpp"
#include "wf_launch.hpp"

namespace wf {

// Pool chunk staging: row r of a chunk starting at pool position p0 is token
// seg[p >> J] 2^J + (p & (2^J - 1)) with p = p0 + r; rows past the end are
// zero.
template <typename T, int D>
struct PoolRows {
  const T* Kunit;
  const int32_t* seg;
  long p0;
  int np, J, mask;
  __device__ __forceinline__ const T* operator()(int r) const {
    if (r >= np) return nullptr;
    const long p = p0 + r;
    const long tok = ((long)seg[p >> J] << J) | (p & mask);
    return Kunit + tok * D;
  }
};

template <int WEIGHTS, typename T, int D>
__global__ __launch_bounds__(kBlock) void scan_chunk_kernel(ScanArgs a) {
  using Stager = RowStager<T, D, kScanChunk, kBlock>;
  constexpr int STRIDE = Stager::STRIDE;
  constexpr int NW = kBlock / kWave;
  constexpr int TB = kScanChunk / 16;       // token blocks per chunk
  constexpr int TBW = TB / NW;              // token blocks per wave
  extern __shared__ __align__(16) unsigned char smem[];
  T* Qs = reinterpret_cast<T*>(smem);                       // [B][STRIDE]
  T* Ks = Qs + (size_t)a.B * STRIDE;                         // [chunk][STRIDE]
  float* red = reinterpret_cast<float*>(Ks + kScanChunk * STRIDE);
  const int nqb = (a.B + 15) / 16;
  // stats pass:   part [nqb][NW][16][2] per chunk, run_m [B], run_z [B]
  // weights pass: row_max [B], row_inv [B]
  float* part = red;
  float* run_m = red + nqb * NW * 32;
  float* run_z = run_m + a.B;

  const int item = xcd_swizzle(blockIdx.x, gridDim.x);
  const int u = item / a.C, c = item % a.C;
  const long pb = (long)c * a.span;
  const long pe = min(pb + (long)a.span, (long)a.P);
  const int nchunks = (int)((pe - pb + kScanChunk - 1) / kScanChunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, col = lane & 15;
  const T* Qunit = reinterpret_cast<const T*>(a.Q) + (long)u * a.B * D;

  PoolRows<T, D> src;
  src.Kunit = reinterpret_cast<const T*>(a.K) + (long)u * a.L * D;
  src.seg = a.seg + (long)u * a.S;
  src.J = a.J;
  src.mask = (1 << a.J) - 1;
  src.p0 = pb;
  src.np = (int)min((long)kScanChunk, pe - pb);
  Stager st;
  st.load(src);

  stage_rows_any<T, D, kBlock>(Qs, a.B, [&](int r) { return Qunit + (long)r * D; });
  if constexpr (WEIGHTS) {
    float* row_max = red;
    float* row_inv = red + a.B;
    const float* stt = a.stats + (long)u * a.C * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      float mx = -INFINITY;
      for (int k = 0; k < a.C; ++k) mx = fmaxf(mx, stt[(long)k * 2 * a.B + q]);
      float z = 0.f;
      for (int k = 0; k < a.C; ++k) {
        const float mk = stt[(long)k * 2 * a.B + q];
        if (mk > -INFINITY) z += stt[(long)k * 2 * a.B + a.B + q] * __expf(mk - mx);
      }
      row_max[q] = mx;
      row_inv[q] = 1.f / z;
    }
  } else {
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      run_m[q] = -INFINITY;
      run_z[q] = 0.f;
    }
  }

  for (int ch = 0; ch < nchunks; ++ch) {
    const long p0 = pb + (long)ch * kScanChunk;
    const int np = (int)min((long)kScanChunk, pe - p0);
    __syncthreads();  // the previous chunk's readers are done with Ks
    st.store(Ks);
    __syncthreads();
    if (ch + 1 < nchunks) {
      src.p0 = p0 + kScanChunk;
      src.np = (int)min((long)kScanChunk, pe - src.p0);
      st.load(src);
    }
    float wacc[TBW];
#pragma unroll
    for (int k = 0; k < TBW; ++k) wacc[k] = 0.f;
    for (int qb = 0; qb < nqb; ++qb) {
      const T* arow = Qs + min(qb * 16 + col, a.B - 1) * STRIDE;
      f32x4 sacc[TBW];
#pragma unroll
      for (int k = 0; k < TBW; ++k) {
        const int tb = wave * TBW + k;
        sacc[k] = tile_dot<T, D>(arow, Ks + (tb * 16 + col) * STRIDE,
                                 f32x4{0.f, 0.f, 0.f, 0.f});
      }
      // lane holds logit[q = 16 qb + 4 g + i][p = p0 + 16 tb + col]
      if constexpr (!WEIGHTS) {
        float* rq = part + (qb * NW + wave) * 32;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float mx = -INFINITY;
#pragma unroll
          for (int k = 0; k < TBW; ++k) {
            const bool ok = (wave * TBW + k) * 16 + col < np;
            const float v = ok ? sacc[k][i] * a.scale : -INFINITY;
            sacc[k][i] = v;
            mx = fmaxf(mx, v);
          }
          mx = wave_max16(mx);
          float z = 0.f;
          if (mx > -INFINITY) {
#pragma unroll
            for (int k = 0; k < TBW; ++k)
              if ((wave * TBW + k) * 16 + col < np) z += __expf(sacc[k][i] - mx);
          }
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) z += __shfl_xor(z, o);
          if (col == 0) {
            rq[(4 * g + i) * 2] = mx;
            rq[(4 * g + i) * 2 + 1] = z;
          }
        }
      } else {
        const float* row_max = red;
        const float* row_inv = red + a.B;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int q = qb * 16 + 4 * g + i;
          if (q < a.B) {
            const float mq = row_max[q], iz = row_inv[q];
#pragma unroll
            for (int k = 0; k < TBW; ++k)
              wacc[k] += __expf(sacc[k][i] * a.scale - mq) * iz;
          }
        }
      }
    }
    if constexpr (!WEIGHTS) {
      __syncthreads();
      for (int q = threadIdx.x; q < a.B; q += kBlock) {
        const int qb = q >> 4, r = q & 15;
        float mx = run_m[q];
#pragma unroll
        for (int w = 0; w < NW; ++w) mx = fmaxf(mx, part[((qb * NW + w) * 16 + r) * 2]);
        float z = run_m[q] > -INFINITY ? run_z[q] * __expf(run_m[q] - mx) : 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const float mw = part[((qb * NW + w) * 16 + r) * 2];
          if (mw > -INFINITY) z += part[((qb * NW + w) * 16 + r) * 2 + 1] * __expf(mw - mx);
        }
        run_m[q] = mx;
        run_z[q] = z;
      }
    } else {
      // column sums over the 4 lane groups (rows 4g + i)
#pragma unroll
      for (int k = 0; k < TBW; ++k) {
        float w = wacc[k];
        w += __shfl_xor(w, 16);
        w += __shfl_xor(w, 32);
        const int pl = (wave * TBW + k) * 16 + col;
        if (g == 0 && pl < np) a.wpool[(long)u * a.P + p0 + pl] = w;
      }
    }
  }
  if constexpr (!WEIGHTS) {
    __syncthreads();
    float* stt = a.stats + ((long)u * a.C + c) * 2 * a.B;
    for (int q = threadIdx.x; q < a.B; q += kBlock) {
      stt[q] = run_m[q];
      stt[a.B + q] = run_z[q];
    }
  }
}

constexpr int kScanSelectBlock = 1024;

__global__ __launch_bounds__(kScanSelectBlock) void scan_select_kernel(
    ScanSelectArgs a, int w_in_lds) {
  __shared__ SelectShared<kScanSelectBlock> sh;
  extern __shared__ float wsh[];
  const int u = blockIdx.x;
  const float* W = a.wpool + (long)u * a.P;
  if (w_in_lds) {
    for (int i = threadIdx.x; i < a.P; i += kScanSelectBlock) wsh[i] = W[i];
    __syncthreads();
  }
  const int32_t* seg = a.seg + (long)u * a.S;
  const int J = a.J;
  const int mask = (1 << J) - 1;
  block_select_topk<kScanSelectBlock>(
      w_in_lds ? wsh : W, a.P, a.keff, a.tok + (long)u * a.keff,
      [=](int p) { return (int32_t)((seg[p >> J] << J) | (p & mask)); }, sh);
}

// ------------------------------------------------------------ host side

ScanPlan plan_scan(const wf_params& p) {
  ScanPlan s;
  const long P = (long)p.segments << p.levels;
  const long U = (long)p.batch * p.heads;
  const long chunks = (P + kScanChunk - 1) / kScanChunk;
  // about 1024 workgroups; each covers 1..8 chunks of the pool
  const long cpw = std::max(1L, std::min(8L, U * chunks / 1024));
  s.span = (int)(cpw * kScanChunk);
  s.chunks = (int)((P + s.span - 1) / s.span);
  const size_t elem = p.dtype == WF_BF16 ? 2 : 4;
  const size_t stride = (size_t)p.head_dim * elem + 16;
  const int nqb = (p.q_len + 15) / 16;
  const size_t red = ((size_t)nqb * 4 * 16 * 2 + (size_t)2 * p.q_len) * sizeof(float);
  s.lds_bytes = (size_t)(p.q_len + kScanChunk) * stride + red;
  return s;
}

template <int WEIGHTS, typename T, int D>
static hipError_t scan_launch(const ScanArgs& a, size_t lds, hipStream_t s) {
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(scan_chunk_kernel<WEIGHTS, T, D>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((scan_chunk_kernel<WEIGHTS, T, D>),
                     dim3((unsigned)(a.U * a.C)), dim3(kBlock), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_scan_chunks(const wf_params& p, int weights, const void* Q,
                              const void* K, const int32_t* seg, float* stats,
                              float* wpool, hipStream_t s) {
  const ScanPlan pl = plan_scan(p);
  ScanArgs a;
  a.Q = Q;
  a.K = K;
  a.seg = seg;
  a.stats = stats;
  a.wpool = wpool;
  a.U = p.batch * p.heads;
  a.L = p.ctx_len;
  a.B = p.q_len;
  a.J = p.levels;
  a.S = p.segments;
  a.P = p.segments << p.levels;
  a.C = pl.chunks;
  a.span = pl.span;
  a.scale = effective_scale(p);
  const bool bf = p.dtype == WF_BF16, d128 = p.head_dim == 128;
  if (weights) {
    if (bf) return d128 ? scan_launch<1, bf16_t, 128>(a, pl.lds_bytes, s)
                        : scan_launch<1, bf16_t, 64>(a, pl.lds_bytes, s);
    return d128 ? scan_launch<1, float, 128>(a, pl.lds_bytes, s)
                : scan_launch<1, float, 64>(a, pl.lds_bytes, s);
  }
  if (bf) return d128 ? scan_launch<0, bf16_t, 128>(a, pl.lds_bytes, s)
                      : scan_launch<0, bf16_t, 64>(a, pl.lds_bytes, s);
  return d128 ? scan_launch<0, float, 128>(a, pl.lds_bytes, s)
              : scan_launch<0, float, 64>(a, pl.lds_bytes, s);
}

hipError_t launch_scan_select(const wf_params& p, const float* wpool,
                              const int32_t* seg, int32_t* tok,
                              hipStream_t s) {
  ScanSelectArgs a;
  a.wpool = wpool;
  a.seg = seg;
  a.tok = tok;
  a.U = p.batch * p.heads;
  a.J = p.levels;
  a.S = p.segments;
  a.P = p.segments << p.levels;
  a.keff = wf_effective_budget(&p);
  const int in_lds = a.P <= kSelectLdsFloats ? 1 : 0;
  const size_t lds = in_lds ? (size_t)a.P * sizeof(float) : 0;
  hipLaunchKernelGGL(scan_select_kernel, dim3((unsigned)a.U),
                     dim3(kScanSelectBlock), lds, s, a, in_lds);
  return hipGetLastError();
}

}  // namespace wf
