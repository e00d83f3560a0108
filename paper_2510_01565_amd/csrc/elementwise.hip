// HBM-bound kernels of the step: adaLN LayerNorm, the modulation GEMV over
// all blocks' adaLN weights, the timestep embedding, the RoPE angle table,
// the Euler update and the V relayout of the stand-alone attention call.
// Rows are processed one per wavefront with 16-byte accesses; all reductions
// are fixed butterfly trees (bitwise deterministic).
#include <math.h>

#include "device_common.h"

namespace dit {

namespace {

// ---------------------------------------------------------------- RoPE table
// table[pos][k] = (cos, sin)(pos * theta^(-2k / (d/2))), evaluated in fp64.
__global__ void rope_table_kernel(float2* table, int quarter, int axis_dim, double theta) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= DIT_MAX_GRID * quarter) return;
  const int pos = i / quarter, k = i % quarter;
  const double ang = (double)pos * pow(theta, -2.0 * k / axis_dim);
  table[i] = make_float2((float)cos(ang), (float)sin(ang));
}

// ---------------------------------------------------------------- timestep embedding
// e[r] = [cos(1000 t f_j) | sin(1000 t f_j)], f_j = 1e4^(-j/half), in fp64.
struct TimeArgs {
  float t[kMaxReq];
};
__global__ void timestep_kernel(float* e, int n_req, TimeArgs ta, int dim) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = dim / 2;
  if (i >= n_req * half) return;
  const int r = i / half, j = i % half;
  const double f = exp(-log(10000.0) * (double)j / half);
  const double ang = 1000.0 * (double)ta.t[r] * f;
  e[(long)r * dim + j] = (float)cos(ang);
  e[(long)r * dim + half + j] = (float)sin(ang);
}

// ---------------------------------------------------------------- GEMV
// y[r, o] = sum_k W[o, k] act(x[r, k]) + b[o] for up to GV_R requests per
// pass; activations staged in LDS, weights streamed once with 16-byte loads.
// Each wavefront takes GemvShape::V output rows at a time and requests all of
// their chunks (a lane holds chunks lane, lane + 64, ... of each row) before
// any arithmetic, so V rows of loads are in flight per wave.  The weights are
// read once per step and never reused, so the loads are nontemporal (they do
// not displace cached data); on MI355X this streams the 6.5 GB of the FLUX
// modulation weights at about 6.8 TB/s against 5.5 TB/s for one row per wave
// with ordinary loads.
constexpr int GV_R = 4;
constexpr int LN_MAX_H = 4096;  // widest hidden size (also the LayerNorm's limit)

template <typename WT>
struct GemvShape {
  static constexpr int EPC = 16 / sizeof(WT);        // elements per 16-byte chunk
  static constexpr int V = sizeof(WT) == 2 ? 4 : 2;  // rows per wave in flight
};

// MAXC: 16-byte chunks per lane and row the registers hold (K <= 64 EPC MAXC)
template <typename WT, int MAXC>
__global__ __launch_bounds__(256) void gemv_kernel(const WT* __restrict__ W, const WT* __restrict__ b,
                                                   const float* __restrict__ x, long ldx, int n_req, int K,
                                                   int N, int act, float* __restrict__ y, long ldy) {
  using S = GemvShape<WT>;
  constexpr int EPC = S::EPC, V = S::V;
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  extern __shared__ float xs[];  // [n_req][K]
  const int nr = min(n_req, GV_R);
  for (int i = threadIdx.x; i < nr * K; i += blockDim.x) {
    const int r = i / K, k = i % K;
    float v = x[(long)r * ldx + k];
    xs[i] = act ? silu(v) : v;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int nwaves = gridDim.x * (blockDim.x >> 6);
  const int chunks = K / EPC;
  // Chunk i of a lane is chunk lane + 64 i of the row; lanes past the row's
  // last chunk load that chunk again (no branch around a load: a branch would
  // end the run of loads in flight) and weigh it by zero.
  int cidx[MAXC];
  float keep[MAXC];
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    cidx[i] = min(lane + 64 * i, chunks - 1);
    keep[i] = lane + 64 * i < chunks ? 1.f : 0.f;
  }
  for (int o0 = (blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)) * V; o0 < N; o0 += nwaves * V) {
    u32x4 u[V][MAXC];
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const u32x4* wr = (const u32x4*)(W + (long)min(o0 + v, N - 1) * K);
#pragma unroll
      for (int i = 0; i < MAXC; ++i) u[v][i] = __builtin_nontemporal_load(wr + cidx[i]);
    }
#pragma unroll
    for (int v = 0; v < V; ++v) {
      float acc[GV_R] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        float wv[EPC];
        if constexpr (sizeof(WT) == 2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            wv[2 * e] = __uint_as_float(u[v][i][e] << 16) * keep[i];
            wv[2 * e + 1] = __uint_as_float(u[v][i][e] & 0xFFFF0000u) * keep[i];
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) wv[e] = __uint_as_float(u[v][i][e]) * keep[i];
        }
#pragma unroll
        for (int r = 0; r < GV_R; ++r) {
          if (r < nr) {
            // 16-byte aligned: K and the chunk offset are multiples of 4 floats
            const float4* xr = (const float4*)(xs + r * K + cidx[i] * EPC);
#pragma unroll
            for (int q = 0; q < EPC / 4; ++q) {
              const float4 xv = xr[q];
              acc[r] = fmaf(wv[4 * q], xv.x, acc[r]);
              acc[r] = fmaf(wv[4 * q + 1], xv.y, acc[r]);
              acc[r] = fmaf(wv[4 * q + 2], xv.z, acc[r]);
              acc[r] = fmaf(wv[4 * q + 3], xv.w, acc[r]);
            }
          }
        }
      }
      const int o = o0 + v;
#pragma unroll
      for (int r = 0; r < GV_R; ++r) {
        if (r < nr) {
          const float sum = wave_sum(acc[r]);
          if (lane == 0 && o < N) y[(long)r * ldy + o] = sum + (b ? to_f32<WT>(b[o]) : 0.f);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- adaLN LayerNorm
// out = LN(x) * (1 + scale[req]) + shift[req], LN with biased variance and no
// affine; statistics in fp32 with a two-pass (mean, then centred squares)
// evaluation from registers.  One wavefront per row, NV float4 per lane
// (H <= 256 NV, at most LN_MAX_H), NV fixed at compile time so the row uses
// no more registers than it needs and more rows stay in flight.

template <typename OT, int NV>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float* __restrict__ X, int H, int row_begin,
                                                     int row_end, const BatchMeta meta,
                                                     const float* __restrict__ mods, int mods_ld, int sh_t,
                                                     int sc_t, int sh_i, int sc_i, float eps, OT* __restrict__ out,
                                                     long ldo) {
  const int lane = threadIdx.x & 63;
  const int R = row_begin + blockIdx.x * 4 + (threadIdx.x >> 6);
  if (R >= row_end) return;
  const int H4 = H >> 2;
  const float4* xr = (const float4*)(X + (long)R * H);
  const RowInfo ri = row_info(meta, R);
  const float* mrow = mods + (long)ri.req * mods_ld;
  const float4* shv = (const float4*)(mrow + (ri.is_img ? sh_i : sh_t));
  const float4* scv = (const float4*)(mrow + (ri.is_img ? sc_i : sc_t));
  // float4 i of a lane is float4 lane + 64 i of the row; lanes past the row
  // load its last float4 again and weigh it by zero (no load behind a branch,
  // so all of them are in flight at once)
  int cidx[NV];
  float keep[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    cidx[i] = min(lane + i * 64, H4 - 1);
    keep[i] = lane + i * 64 < H4 ? 1.f : 0.f;
  }
  float4 v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = xr[cidx[i]];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) s += keep[i] * ((v[i].x + v[i].y) + (v[i].z + v[i].w));
  const float mean = wave_sum(s) / (float)H;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i].x -= mean;
    v[i].y -= mean;
    v[i].z -= mean;
    v[i].w -= mean;
    ss += keep[i] * ((v[i].x * v[i].x + v[i].y * v[i].y) + (v[i].z * v[i].z + v[i].w * v[i].w));
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / (float)H + eps);
  OT* orow = out + (long)(R - row_begin) * ldo;
  // Every lane stores: a lane past the row's end writes the row's last
  // float4 with exactly the bytes the lane that owns it writes (same inputs,
  // same arithmetic), so no store needs a branch and the shift / scale loads
  // all leave before the first store.
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = cidx[i];
    const float4 sh = shv[c], sc = scv[c];
    const float y0 = v[i].x * rstd * (1.f + sc.x) + sh.x;
    const float y1 = v[i].y * rstd * (1.f + sc.y) + sh.y;
    const float y2 = v[i].z * rstd * (1.f + sc.z) + sh.z;
    const float y3 = v[i].w * rstd * (1.f + sc.w) + sh.w;
    if constexpr (sizeof(OT) == 2) {
      uint2 w;
      w.x = pack_bf16x2(y0, y1);
      w.y = pack_bf16x2(y2, y3);
      *(uint2*)(orow + c * 4) = w;
    } else {
      *(float4*)(orow + c * 4) = make_float4(y0, y1, y2, y3);
    }
  }
}

// ---------------------------------------------------------------- Euler
struct DtArgs {
  float dt[kMaxReq];
};
template <typename T>
__global__ void euler_kernel(T* __restrict__ x, const T* __restrict__ v, long n, int channels, const BatchMeta meta,
                             DtArgs da) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int row = (int)(i / channels);
  int r = 0;
  while (r + 1 < meta.n_req && row >= meta.img_off[r + 1]) ++r;
  const float xv = to_f32<T>(x[i]), vv = to_f32<T>(v[i]);
  x[i] = from_f32<T>(xv - da.dt[r] * vv);
}

// ---------------------------------------------------------------- V relayout
template <typename T>
__global__ void v_transpose_kernel(const T* __restrict__ v, const BatchMeta meta, int heads, int d,
                                   T* __restrict__ vt, long ld) {
  __shared__ T tile[32][33];
  const int h = blockIdx.z;
  const int p0 = blockIdx.x * 32, d0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  const int T_ = meta.T;
  for (int yy = ty; yy < 32; yy += 8) {
    const int p = p0 + yy, dd = d0 + tx;
    if (p < T_ && dd < d) tile[yy][tx] = v[((long)p * heads + h) * d + dd];
  }
  __syncthreads();
  for (int yy = ty; yy < 32; yy += 8) {
    const int dd = d0 + yy, p = p0 + tx;
    if (p < T_ && dd < d) {
      int r = 0;
      while (r + 1 < meta.n_req && p >= meta.joint_off[r + 1]) ++r;
      const int col = vt_slot(meta.pad_off[r] + (p - meta.joint_off[r]));
      vt[((long)h * d + dd) * ld + col] = tile[tx][yy];
    }
  }
}

template <typename T>
__global__ void vt_pad_zero_kernel(T* __restrict__ vt, const BatchMeta meta, long ld) {
  const long row = blockIdx.x;  // h * d + dd
  for (int r = 0; r < meta.n_req; ++r) {
    const int L = meta.joint_off[r + 1] - meta.joint_off[r];
    const int P = meta.pad_off[r + 1] - meta.pad_off[r];
    for (int k = L + threadIdx.x; k < P; k += blockDim.x) vt[row * ld + vt_slot(meta.pad_off[r] + k)] = T(0);
  }
}

}  // namespace

namespace {
__global__ void zero_i32_kernel(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}
}  // namespace

hipError_t launch_zero_i32(int* p, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_i32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_vt_pad_zero(int dtype, void* vt, long ld, const BatchMeta& meta, int heads, int d, hipStream_t s) {
  const dim3 grid((unsigned)(heads * d));
  if (dtype == DIT_BF16)
    hipLaunchKernelGGL(vt_pad_zero_kernel<bf16_t>, grid, dim3(64), 0, s, (bf16_t*)vt, meta, ld);
  else
    hipLaunchKernelGGL(vt_pad_zero_kernel<float>, grid, dim3(64), 0, s, (float*)vt, meta, ld);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* table, int head_dim, float theta, hipStream_t s) {
  const int quarter = head_dim / 4;
  const int n = DIT_MAX_GRID * quarter;
  hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, s, table, quarter, head_dim / 2,
                     (double)theta);
  return hipGetLastError();
}

hipError_t launch_timestep_embed(float* e, int n_req, const float* t_host, int dim, hipStream_t s) {
  TimeArgs ta{};
  for (int r = 0; r < n_req; ++r) ta.t[r] = t_host[r];
  const int n = n_req * (dim / 2);
  hipLaunchKernelGGL(timestep_kernel, dim3((n + 255) / 256), dim3(256), 0, s, e, n_req, ta, dim);
  return hipGetLastError();
}

template <typename WT, int MAXC>
void gemv_launch(int blocks, size_t shmem, hipStream_t s, const void* W, const void* b, const float* x, long ldx,
                 int nr, int K, int N, int act, float* y, long ldy) {
  hipLaunchKernelGGL((gemv_kernel<WT, MAXC>), dim3(blocks), dim3(256), shmem, s, (const WT*)W, (const WT*)b, x, ldx,
                     nr, K, N, act, y, ldy);
}

template <typename WT>
void gemv_dispatch(int blocks, size_t shmem, hipStream_t s, const void* W, const void* b, const float* x, long ldx,
                   int nr, int K, int N, int act, float* y, long ldy) {
  const int c = (K / GemvShape<WT>::EPC + 63) / 64;  // chunks per lane and row
  if (c <= 1) gemv_launch<WT, 1>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else if (c <= 2) gemv_launch<WT, 2>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else if (c <= 3) gemv_launch<WT, 3>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else if (c <= 4) gemv_launch<WT, 4>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else if (c <= 6) gemv_launch<WT, 6>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else if (c <= 8) gemv_launch<WT, 8>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
  else gemv_launch<WT, 16>(blocks, shmem, s, W, b, x, ldx, nr, K, N, act, y, ldy);
}

hipError_t launch_gemv(int wdtype, const void* W, const void* b, const float* x, long ldx, int n_req, int K,
                       int N, int act, float* y, long ldy, hipStream_t s) {
  if (K > LN_MAX_H) return hipErrorInvalidValue;
  const size_t shmem = (size_t)(n_req < GV_R ? n_req : GV_R) * K * sizeof(float);
  const int V = wdtype == DIT_BF16 ? GemvShape<bf16_t>::V : GemvShape<float>::V;
  int blocks = (N + 4 * V - 1) / (4 * V);
  if (blocks > 256 * 32) blocks = 256 * 32;
  for (int r0 = 0; r0 < n_req; r0 += GV_R) {
    const int nr = n_req - r0 < GV_R ? n_req - r0 : GV_R;
    if (wdtype == DIT_BF16)
      gemv_dispatch<bf16_t>(blocks, shmem, s, W, b, x + (long)r0 * ldx, ldx, nr, K, N, act, y + (long)r0 * ldy, ldy);
    else
      gemv_dispatch<float>(blocks, shmem, s, W, b, x + (long)r0 * ldx, ldx, nr, K, N, act, y + (long)r0 * ldy, ldy);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_ln_modulate(int out_dtype, const float* X, int H, int row_begin, int row_end,
                              const BatchMeta& meta, const float* mods, int mods_ld, int shift_txt, int scale_txt,
                              int shift_img, int scale_img, float eps, void* out, long ldo, hipStream_t s) {
  const int rows = row_end - row_begin;
  if (rows <= 0) return hipSuccess;
  if (H > LN_MAX_H) return hipErrorInvalidValue;
  const dim3 grid((rows + 3) / 4);
  const int nv = (H / 4 + 63) / 64;
#define DIT_LN_LAUNCH(OT, NV)                                                                                 \
  hipLaunchKernelGGL((ln_mod_kernel<OT, NV>), grid, dim3(256), 0, s, X, H, row_begin, row_end, meta, mods, mods_ld, \
                     shift_txt, scale_txt, shift_img, scale_img, eps, (OT*)out, ldo)
#define DIT_LN_DISPATCH(OT)          \
  if (nv <= 2) DIT_LN_LAUNCH(OT, 2);  \
  else if (nv <= 4) DIT_LN_LAUNCH(OT, 4); \
  else if (nv <= 8) DIT_LN_LAUNCH(OT, 8); \
  else if (nv <= 12) DIT_LN_LAUNCH(OT, 12); \
  else DIT_LN_LAUNCH(OT, 16);
  if (out_dtype == DIT_BF16) {
    DIT_LN_DISPATCH(bf16_t)
  } else {
    DIT_LN_DISPATCH(float)
  }
#undef DIT_LN_DISPATCH
#undef DIT_LN_LAUNCH
  return hipGetLastError();
}

hipError_t launch_euler(int dtype, void* x, const void* v, int channels, const BatchMeta& meta,
                        const float* dt_host, hipStream_t s) {
  DtArgs da{};
  for (int r = 0; r < meta.n_req; ++r) da.dt[r] = dt_host[r];
  const long n = (long)meta.T_img * channels;
  if (n == 0) return hipSuccess;
  const dim3 grid((unsigned)((n + 255) / 256));
  if (dtype == DIT_BF16)
    hipLaunchKernelGGL(euler_kernel<bf16_t>, grid, dim3(256), 0, s, (bf16_t*)x, (const bf16_t*)v, n, channels, meta,
                       da);
  else
    hipLaunchKernelGGL(euler_kernel<float>, grid, dim3(256), 0, s, (float*)x, (const float*)v, n, channels, meta,
                       da);
  return hipGetLastError();
}

hipError_t launch_v_transpose(int dtype, const void* v, const BatchMeta& meta, int heads, int d, void* vt,
                              hipStream_t s) {
  const long ld = meta.pad_off[meta.n_req];
  const dim3 grid((meta.T + 31) / 32, (d + 31) / 32, heads);
  if (meta.T == 0) return hipSuccess;
  if (dtype == DIT_BF16)
    hipLaunchKernelGGL(v_transpose_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)v, meta, heads, d,
                       (bf16_t*)vt, ld);
  else
    hipLaunchKernelGGL(v_transpose_kernel<float>, grid, dim3(256), 0, s, (const float*)v, meta, heads, d, (float*)vt,
                       ld);
  return hipGetLastError();
}

}  // namespace dit
