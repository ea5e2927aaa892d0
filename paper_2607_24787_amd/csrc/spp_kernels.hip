// gfx950 kernels of the offloaded-MoE decode hot path.
//
// Lane layout shared by every row-dot kernel: a row of D elements is read as
// 16-byte chunks (8 bf16 or 4 fp32); lane l of a 64-wide wave owns chunks
// l, l+64, l+128, ... so one wave-wide load instruction moves 1 KiB of
// contiguous memory.  A row's dot product is the sum of per-lane partial sums
// followed by a butterfly reduction across the wave (every lane ends with the
// same bits, since fp32 addition is commutative).
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstdint>

#include "spp_internal.h"

namespace spp {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

template <typename T>
struct Vec;
template <>
struct Vec<float> {
  static constexpr int N = 4;
};
template <>
struct Vec<uint16_t> {
  static constexpr int N = 8;
};

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

template <typename T>
__device__ __forceinline__ void unpack(const uint4 r, float* f);
template <>
__device__ __forceinline__ void unpack<float>(const uint4 r, float* f) {
  f[0] = __uint_as_float(r.x);
  f[1] = __uint_as_float(r.y);
  f[2] = __uint_as_float(r.z);
  f[3] = __uint_as_float(r.w);
}
template <>
__device__ __forceinline__ void unpack<uint16_t>(const uint4 r, float* f) {
  f[0] = __uint_as_float(r.x << 16);
  f[1] = __uint_as_float(r.x & 0xffff0000u);
  f[2] = __uint_as_float(r.y << 16);
  f[3] = __uint_as_float(r.y & 0xffff0000u);
  f[4] = __uint_as_float(r.z << 16);
  f[5] = __uint_as_float(r.z & 0xffff0000u);
  f[6] = __uint_as_float(r.w << 16);
  f[7] = __uint_as_float(r.w & 0xffff0000u);
}

template <typename T>
__device__ __forceinline__ float load_elem(const void* p, size_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const void* p, size_t i) {
  return reinterpret_cast<const float*>(p)[i];
}
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const void* p, size_t i) {
  return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(p)[i]) << 16);
}

template <typename T>
__device__ __forceinline__ void store_elem(void* p, size_t i, float v);
template <>
__device__ __forceinline__ void store_elem<float>(void* p, size_t i, float v) {
  reinterpret_cast<float*>(p)[i] = v;
}
template <>
__device__ __forceinline__ void store_elem<uint16_t>(void* p, size_t i, float v) {
  // round to nearest, ties to even
  uint32_t b = __float_as_uint(v);
  uint16_t o;
  if ((b & 0x7fffffffu) > 0x7f800000u) {
    o = 0x7fc0;  // NaN
  } else {
    b += 0x7fffu + ((b >> 16) & 1u);
    o = static_cast<uint16_t>(b >> 16);
  }
  reinterpret_cast<uint16_t*>(p)[i] = o;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Row of D input values of token b in lane layout, as fp32.
template <typename T, int NCH>
__device__ __forceinline__ void load_row_f32(const float* src, int lane, int nch, float (&xv)[NCH][Vec<T>::N]) {
  constexpr int V = Vec<T>::N;
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = lane + 64 * j;
#pragma unroll
    for (int v = 0; v < V; ++v) xv[j][v] = 0.f;
    if (c < nch) {
#pragma unroll
      for (int v = 0; v < V; v += 4) {
        const uint4 r = ld16(src + c * V + v);
        unpack<float>(r, &xv[j][v]);
      }
    }
  }
}

template <typename T, int NCH>
__device__ __forceinline__ void load_row_storage(const T* src, int lane, int nch, float (&xv)[NCH][Vec<T>::N]) {
  constexpr int V = Vec<T>::N;
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = lane + 64 * j;
#pragma unroll
    for (int v = 0; v < V; ++v) xv[j][v] = 0.f;
    if (c < nch) unpack<T>(ld16(src + c * V), xv[j]);
  }
}

template <typename T, int NCH>
__device__ __forceinline__ float rms_scale(float (&xv)[NCH][Vec<T>::N], int D, float eps) {
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NCH; ++j)
#pragma unroll
    for (int v = 0; v < Vec<T>::N; ++v) ss += xv[j][v] * xv[j][v];
  ss = wave_sum(ss);
  return 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
}

// ---------------------------------------------------------------------------
// Router logits, adapter hidden units, then (last workgroup) Top-K, gates and
// adapter priorities.  One wave per weight row.
// ---------------------------------------------------------------------------
template <typename T, int NCH>
__global__ __launch_bounds__(kThreads) void router_adapter_kernel(RouterArgs a) {
  constexpr int V = Vec<T>::N;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = a.D, nch = D / V, n = a.n, r = a.r, ldz = a.n + a.r;
  const int nr = a.router_on ? n : 0;
  const int na = a.A ? r : 0;
  const int row = blockIdx.x * kWaves + wave;

  __shared__ int s_last;
  __shared__ float s_zsel[kWaves][32];
  __shared__ int s_isel[kWaves][32];
  __shared__ float s_red[kWaves];
  __shared__ float s_a[256];

  const T* wrow = nullptr;
  int zcol = 0;
  if (row < nr) {
    wrow = reinterpret_cast<const T*>(a.Wr) + static_cast<size_t>(row) * D;
    zcol = row;
  } else if (row < nr + na) {
    wrow = reinterpret_cast<const T*>(a.A) + static_cast<size_t>(row - nr) * D;
    zcol = n + (row - nr);
  }
  uint4 w[NCH];
  if (wrow) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int c = lane + 64 * j;
      w[j] = c < nch ? ld16(wrow + c * V) : make_uint4(0, 0, 0, 0);
    }
  }

  for (int b = 0; b < a.B; ++b) {
    float xv[NCH][V];
    if (a.u) {
      load_row_f32<T, NCH>(a.u + static_cast<size_t>(b) * D, lane, nch, xv);
    } else {
      load_row_storage<T, NCH>(reinterpret_cast<const T*>(a.h) + static_cast<size_t>(b) * D, lane, nch, xv);
    }
    if (!a.x_given) {
      const float inv = rms_scale<T, NCH>(xv, D, a.eps);
#pragma unroll
      for (int j = 0; j < NCH; ++j)
#pragma unroll
        for (int v = 0; v < V; ++v) xv[j][v] *= inv;
    }
    if (blockIdx.x == 0 && wave == 0 && a.x_out) {
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) {
          float* dst = a.x_out + static_cast<size_t>(b) * D + c * V;
#pragma unroll
          for (int v = 0; v < V; ++v) dst[v] = xv[j][v];
        }
      }
    }
    if (wrow) {
      float acc = 0.f;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        float wf[V];
        unpack<T>(w[j], wf);
#pragma unroll
        for (int v = 0; v < V; ++v) acc += wf[v] * xv[j][v];
      }
      acc = wave_sum(acc);
      if (lane == 0) st_agent(a.zbuf + static_cast<size_t>(b) * ldz + zcol, acc);
    }
  }

  // single-pass handoff: the last workgroup to finish does the selection
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(a.counter, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == gridDim.x - 1);
  }
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  if (a.router_on) {
    constexpr int QMAX = kMaxExpertsTopK / 64;
    const int nq = (n + 63) / 64;
    for (int b = wave; b < a.B; b += kWaves) {
      const float* zb = a.zbuf + static_cast<size_t>(b) * ldz;
      float v[QMAX];
      uint32_t used = 0;
#pragma unroll
      for (int q = 0; q < QMAX; ++q) {
        const int e = lane + 64 * q;
        v[q] = (q < nq && e < n) ? ld_agent(zb + e) : -INFINITY;
      }
      for (int k = 0; k < a.K; ++k) {
        float bv = -INFINITY;
        int bi = INT_MAX;
#pragma unroll
        for (int q = 0; q < QMAX; ++q) {
          const int e = lane + 64 * q;
          if (q < nq && e < n && !((used >> q) & 1u)) {
            if (v[q] > bv || (v[q] == bv && e < bi)) {
              bv = v[q];
              bi = e;
            }
          }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
          const float ov = __shfl_xor(bv, o, 64);
          const int oi = __shfl_xor(bi, o, 64);
          if (ov > bv || (ov == bv && oi < bi)) {
            bv = ov;
            bi = oi;
          }
        }
        if (bi != INT_MAX && (bi & 63) == lane) used |= 1u << (bi >> 6);
        if (lane == 0) {
          s_zsel[wave][k] = bv;
          s_isel[wave][k] = bi;
        }
      }
      if (lane == 0) {
        // softmax over all n renormalised over the K selected = softmax over the selected
        const float m = s_zsel[wave][0];
        float sum = 0.f;
        for (int k = 0; k < a.K; ++k) {
          const float e = expf(s_zsel[wave][k] - m);
          s_zsel[wave][k] = e;
          sum += e;
        }
        for (int k = 0; k < a.K; ++k) {
          a.topk[b * a.K + k] = s_isel[wave][k];
          a.gates[b * a.K + k] = s_zsel[wave][k] / sum;
        }
      }
    }
  }

  if (na) {
    // z_hat = B a per token, softmax over the n experts, summed over tokens in order
    constexpr int EQ = kMaxExpertsTopK / kThreads;
    float sacc[EQ];
#pragma unroll
    for (int q = 0; q < EQ; ++q) sacc[q] = 0.f;
    for (int b = 0; b < a.B; ++b) {
      __syncthreads();
      for (int j = threadIdx.x; j < r; j += kThreads) s_a[j] = ld_agent(a.zbuf + static_cast<size_t>(b) * ldz + n + j);
      __syncthreads();
      float zh[EQ];
      float mx = -INFINITY;
#pragma unroll
      for (int q = 0; q < EQ; ++q) {
        const int e = threadIdx.x + kThreads * q;
        zh[q] = -INFINITY;
        if (e < n) {
          float acc = 0.f;
          for (int j = 0; j < r; ++j) acc += load_elem<T>(a.Bm, static_cast<size_t>(e) * r + j) * s_a[j];
          zh[q] = acc;
          mx = fmaxf(mx, acc);
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      if (lane == 0) s_red[wave] = mx;
      __syncthreads();
      mx = s_red[0];
      for (int wv = 1; wv < kWaves; ++wv) mx = fmaxf(mx, s_red[wv]);
      __syncthreads();
      float ex[EQ];
      float part = 0.f;
#pragma unroll
      for (int q = 0; q < EQ; ++q) {
        const int e = threadIdx.x + kThreads * q;
        ex[q] = e < n ? expf(zh[q] - mx) : 0.f;
        part += ex[q];
      }
      part = wave_sum(part);
      if (lane == 0) s_red[wave] = part;
      __syncthreads();
      float sum = 0.f;
      for (int wv = 0; wv < kWaves; ++wv) sum += s_red[wv];
#pragma unroll
      for (int q = 0; q < EQ; ++q) sacc[q] += ex[q] / sum;
    }
#pragma unroll
    for (int q = 0; q < EQ; ++q) {
      const int e = threadIdx.x + kThreads * q;
      if (e < n) a.s[e] = sacc[q];
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(a.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Routed-expert SwiGLU FFN, one pass over the expert blobs.  The work is the
// flat list of (expert, unit i) pairs; unit i of an expert is the contiguous
// [gate row i | up row i | down column i].  A wave computes
//   h_i = silu(gate_i . x) * (up_i . x) * g_k
// and accumulates h_i * down_i into its lane-owned slice of y; the workgroup
// then sums its waves and writes one partial y.
// ---------------------------------------------------------------------------
template <typename T, int NCH>
__global__ __launch_bounds__(kThreads) void ffn_units_kernel(FfnArgs a) {
  constexpr int V = Vec<T>::N;
  extern __shared__ float s_red[];  // [kWaves][D]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = a.D, nch = D / V, I = a.I;

  float xv[NCH][V];
  load_row_f32<T, NCH>(a.x, lane, nch, xv);
  float acc[NCH][V];
#pragma unroll
  for (int j = 0; j < NCH; ++j)
#pragma unroll
    for (int v = 0; v < V; ++v) acc[j][v] = 0.f;

  const int total = a.nW * I;
  const int u0 = blockIdx.x * a.upw;
  const int u1 = min(u0 + a.upw, total);
  const size_t unit_elems = static_cast<size_t>(3) * D;

  int uidx = u0 + wave;
  // two units per iteration keep 6*NCH 16-byte loads in flight per lane
  for (; uidx + kWaves < u1; uidx += 2 * kWaves) {
    uint4 rg[2][NCH], ru[2][NCH], rd[2][NCH];
    float gate[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int uu = uidx + p * kWaves;
      const int d = uu / I, i = uu - d * I;
      const T* base = reinterpret_cast<const T*>(a.blob[d]) + static_cast<size_t>(i) * unit_elems;
      gate[p] = a.gate_idx[d] >= 0 ? a.gates[a.gate_idx[d]] : 1.f;
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int c = lane + 64 * j;
        if (c < nch) {
          rg[p][j] = ld16(base + c * V);
          ru[p][j] = ld16(base + D + c * V);
          rd[p][j] = ld16(base + 2 * D + c * V);
        } else {
          rg[p][j] = ru[p][j] = rd[p][j] = make_uint4(0, 0, 0, 0);
        }
      }
    }
    float gs[2] = {0.f, 0.f}, us[2] = {0.f, 0.f};
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        float fg[V], fu[V];
        unpack<T>(rg[p][j], fg);
        unpack<T>(ru[p][j], fu);
#pragma unroll
        for (int v = 0; v < V; ++v) {
          gs[p] += fg[v] * xv[j][v];
          us[p] += fu[v] * xv[j][v];
        }
      }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      gs[0] += __shfl_xor(gs[0], o, 64);
      us[0] += __shfl_xor(us[0], o, 64);
      gs[1] += __shfl_xor(gs[1], o, 64);
      us[1] += __shfl_xor(us[1], o, 64);
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const float hval = gs[p] / (1.f + expf(-gs[p])) * us[p] * gate[p];
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        float fd[V];
        unpack<T>(rd[p][j], fd);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[j][v] += hval * fd[v];
      }
    }
  }
  for (; uidx < u1; uidx += kWaves) {
    const int d = uidx / I, i = uidx - d * I;
    const T* base = reinterpret_cast<const T*>(a.blob[d]) + static_cast<size_t>(i) * unit_elems;
    const float gate = a.gate_idx[d] >= 0 ? a.gates[a.gate_idx[d]] : 1.f;
    uint4 rg[NCH], ru[NCH], rd[NCH];
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int c = lane + 64 * j;
      if (c < nch) {
        rg[j] = ld16(base + c * V);
        ru[j] = ld16(base + D + c * V);
        rd[j] = ld16(base + 2 * D + c * V);
      } else {
        rg[j] = ru[j] = rd[j] = make_uint4(0, 0, 0, 0);
      }
    }
    float gs = 0.f, us = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      float fg[V], fu[V];
      unpack<T>(rg[j], fg);
      unpack<T>(ru[j], fu);
#pragma unroll
      for (int v = 0; v < V; ++v) {
        gs += fg[v] * xv[j][v];
        us += fu[v] * xv[j][v];
      }
    }
    gs = wave_sum(gs);
    us = wave_sum(us);
    const float hval = gs / (1.f + expf(-gs)) * us * gate;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      float fd[V];
      unpack<T>(rd[j], fd);
#pragma unroll
      for (int v = 0; v < V; ++v) acc[j][v] += hval * fd[v];
    }
  }

  // sum the waves of this workgroup, wave order fixed
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = lane + 64 * j;
    if (c < nch) {
#pragma unroll
      for (int v = 0; v < V; ++v) s_red[wave * D + c * V + v] = acc[j][v];
    }
  }
  __syncthreads();
  float* out = a.partial + static_cast<size_t>(blockIdx.x) * D;
  for (int d = threadIdx.x; d < D; d += kThreads) {
    float s = s_red[d];
#pragma unroll
    for (int wv = 1; wv < kWaves; ++wv) s += s_red[wv * D + d];
    out[d] = s;
  }
}

// y = sum of the workgroup partials (fixed order), h_out = round(residual + y).
// 256 threads cover 64 outputs: four groups split the partials, then combine.
template <typename T>
__global__ __launch_bounds__(kThreads) void ffn_combine_kernel(CombineArgs a) {
  __shared__ float s_part[kWaves][64];
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (col < a.D)
    for (int w = grp; w < a.nparts; w += kWaves) s += a.partial[static_cast<size_t>(w) * a.D + col];
  s_part[grp][lane] = s;
  __syncthreads();
  if (grp == 0 && col < a.D) {
    const float y = ((s_part[0][lane] + s_part[1][lane]) + s_part[2][lane]) + s_part[3][lane];
    const float res = a.res_u ? a.res_u[col] : load_elem<T>(a.res_h, col);
    store_elem<T>(a.out, col, res + y);
  }
}

// Stand-in projection prologue: u = h + P rms(h) (fp32 result).  One wave per row of P.
template <typename T, int NCH>
__global__ __launch_bounds__(kThreads) void proj_kernel(ProjArgs a) {
  constexpr int V = Vec<T>::N;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int D = a.D, nch = D / V;
  const int row = blockIdx.x * kWaves + wave;
  if (row >= D) return;
  const T* prow = reinterpret_cast<const T*>(a.P) + static_cast<size_t>(row) * D;
  uint4 w[NCH];
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int c = lane + 64 * j;
    w[j] = c < nch ? ld16(prow + c * V) : make_uint4(0, 0, 0, 0);
  }
  for (int b = 0; b < a.B; ++b) {
    const T* hb = reinterpret_cast<const T*>(a.h) + static_cast<size_t>(b) * D;
    float xv[NCH][V];
    load_row_storage<T, NCH>(hb, lane, nch, xv);
    const float inv = rms_scale<T, NCH>(xv, D, a.eps);
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      float wf[V];
      unpack<T>(w[j], wf);
#pragma unroll
      for (int v = 0; v < V; ++v) acc += wf[v] * (xv[j][v] * inv);
    }
    acc = wave_sum(acc);
    if (lane == 0) a.u[static_cast<size_t>(b) * D + row] = load_elem<T>(hb, row) + acc;
  }
}

template <typename T>
int nch_for(int D) {
  const int nch = D / Vec<T>::N;
  return (nch + 63) / 64;
}

#define SPP_DISPATCH_NCH(NCHV, ...)                          \
  switch (NCHV) {                                            \
    case 1: { constexpr int NCH = 1; __VA_ARGS__; } break;   \
    case 2: { constexpr int NCH = 2; __VA_ARGS__; } break;   \
    case 3: { constexpr int NCH = 3; __VA_ARGS__; } break;   \
    case 4: { constexpr int NCH = 4; __VA_ARGS__; } break;   \
    case 5: { constexpr int NCH = 5; __VA_ARGS__; } break;   \
    case 6: { constexpr int NCH = 6; __VA_ARGS__; } break;   \
    case 7: { constexpr int NCH = 7; __VA_ARGS__; } break;   \
    case 8: { constexpr int NCH = 8; __VA_ARGS__; } break;   \
    default: return hipErrorInvalidValue;                    \
  }

template <typename T>
hipError_t router_t(const RouterArgs& a, hipStream_t st) {
  const int rows = (a.router_on ? a.n : 0) + (a.A ? a.r : 0);
  if (rows <= 0) return hipErrorInvalidValue;
  const int grid = (rows + kWaves - 1) / kWaves;
  SPP_DISPATCH_NCH(nch_for<T>(a.D),
                   hipLaunchKernelGGL((router_adapter_kernel<T, NCH>), dim3(grid), dim3(kThreads), 0, st, a));
  return hipGetLastError();
}

template <typename T>
hipError_t ffn_t(const FfnArgs& a, int grid, hipStream_t st) {
  const size_t lds = sizeof(float) * kWaves * a.D;
  SPP_DISPATCH_NCH(nch_for<T>(a.D),
                   hipLaunchKernelGGL((ffn_units_kernel<T, NCH>), dim3(grid), dim3(kThreads), lds, st, a));
  return hipGetLastError();
}

template <typename T>
hipError_t proj_t(const ProjArgs& a, hipStream_t st) {
  const int grid = (a.D + kWaves - 1) / kWaves;
  SPP_DISPATCH_NCH(nch_for<T>(a.D),
                   hipLaunchKernelGGL((proj_kernel<T, NCH>), dim3(grid), dim3(kThreads), 0, st, a));
  return hipGetLastError();
}

int g_ffn_target_wgs = 256;

}  // namespace

hipError_t launch_router(const RouterArgs& a, int dtype, hipStream_t st) {
  if (a.n > kMaxExpertsTopK || a.r > 256 || a.K > 32 || a.K > a.n) return hipErrorInvalidValue;
  return dtype == 1 ? router_t<uint16_t>(a, st) : router_t<float>(a, st);
}

hipError_t launch_ffn(const FfnArgs& a, int grid, int dtype, hipStream_t st) {
  if (a.nW <= 0 || a.nW > kMaxWork || grid <= 0) return hipErrorInvalidValue;
  return dtype == 1 ? ffn_t<uint16_t>(a, grid, st) : ffn_t<float>(a, grid, st);
}

hipError_t launch_combine(const CombineArgs& a, int dtype, hipStream_t st) {
  const int grid = (a.D + 63) / 64;
  if (dtype == 1)
    hipLaunchKernelGGL((ffn_combine_kernel<uint16_t>), dim3(grid), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((ffn_combine_kernel<float>), dim3(grid), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_proj(const ProjArgs& a, int dtype, hipStream_t st) {
  return dtype == 1 ? proj_t<uint16_t>(a, st) : proj_t<float>(a, st);
}

void set_ffn_target_wgs(int wgs) { g_ffn_target_wgs = wgs > 0 ? wgs : 256; }

// Units per workgroup so that about g_ffn_target_wgs workgroups share the work.
int ffn_grid_for(int nunits, int* upw) {
  int grid = (nunits + kWaves - 1) / kWaves;
  if (grid > g_ffn_target_wgs) grid = g_ffn_target_wgs;
  if (grid < 1) grid = 1;
  *upw = (nunits + grid - 1) / grid;
  return (nunits + *upw - 1) / *upw;
}

size_t ffn_max_grid() { return 4096; }


}  // namespace spp
