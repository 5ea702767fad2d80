// Shared projections (a3, a7, a9, a10): ONE GEMM over every row of the mixed
// batch, C[m, n] = sum_k X[m, k] W[n, k], with the per-task LoRA expand fused
// in as extra MFMA steps and the bias / activation / residual fused into the
// epilogue.
//
// The paper batches all requests through the shared backbone and then adds
// each adapter's difference on its own requests (Section 4.2, adapter
// handling; Fig. 5 (c)).  Here the difference is not a second pass over the
// output: after the K loop, a tile that holds rows of tasks t0..t1 (rows are
// sorted by task, so a tile spans a contiguous task range) runs, per task,
// ceil(r_t / 32) more MFMA steps with A-operand B_t (the task's expand factor,
// read straight from its device pointer) and B-operand U (the per-row shrink
// output s_t x A_t^T), masked to that task's rows.  The sum is exactly
// x W^T + s_t (x A_t^T) B_t^T per row.
//
// bf16 path (gfx950): v_mfma_f32_16x16x32_bf16, 128x128x64 block tile,
// 4 waves of 64x64, LDS double buffer with an XOR swizzle so that both the
// 16-byte fragment reads and the row writes are bank-conflict free, global
// loads for tile k+1 in flight during the MFMAs of tile k.  The weight tile
// feeds the MFMA A slot and the activation tile the B slot, so each lane ends
// up with 4 consecutive output columns of one row: epilogue stores are 8-byte
// (bf16) or 16-byte (fp32) vectors.
//
// fp32 path: a plain LDS-tiled FMA GEMM with the same epilogues (the tiny
// fp32 encoder workload only needs exactness, not speed).
#include "vfm_internal.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;

__device__ __forceinline__ int swz(int row, int kc) { return kc ^ ((row & 7) ^ ((row >> 3) & 1)); }

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.f + erff(v * 0.70710678118654752440f));
}
__device__ __forceinline__ float silu_f(float v) { return v / (1.f + expf(-v)); }

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int EPI, bool SWIGLU>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * BK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int NT = SWIGLU ? BN / 2 : BN;  // output columns per block
  const int n_tiles_n = (a.N + NT - 1) / NT;
  const int tn = blockIdx.x % n_tiles_n, tm = blockIdx.x / n_tiles_n;
  const int m0 = tm * BM, n0 = tn * NT;
  const bf16* X = (const bf16*)a.X;
  const bf16* W = (const bf16*)a.W;
  const bf16* W2 = (const bf16*)a.W2;

  const bf16* xsrc[4];
  const bf16* wsrc[4];
  int lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    const int m = min(m0 + row, a.M - 1);
    xsrc[i] = X + (int64_t)m * a.ldx + kc * 8;
    const bf16* wb = W;
    int wrow;
    if (SWIGLU) {
      const int sub = row >> 4;
      wb = (sub & 1) ? W2 : W;
      wrow = min(n0 + (sub >> 1) * 16 + (row & 15), a.N - 1);
    } else {
      wrow = min(n0 + row, a.N - 1);
    }
    wsrc[i] = wb + (int64_t)wrow * a.K + kc * 8;
    lds_off[i] = row * BK + swz(row, kc) * 8;
  }

  bf16x8 xr[4], wr[4];
  f32x4 acc[4][4];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = a.K / BK;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    xr[i] = *reinterpret_cast<const bf16x8*>(xsrc[i]);
    wr[i] = *reinterpret_cast<const bf16x8*>(wsrc[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<bf16x8*>(&As[0][lds_off[i]]) = xr[i];
    *reinterpret_cast<bf16x8*>(&Bs[0][lds_off[i]]) = wr[i];
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) {
      const int k0 = (kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xr[i] = *reinterpret_cast<const bf16x8*>(xsrc[i] + k0);
        wr[i] = *reinterpret_cast<const bf16x8*>(wsrc[i] + k0);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kc = kk * 4 + (lane >> 4);
      bf16x8 wf[4], xf[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int r = wn * 64 + ni * 16 + (lane & 15);
        wf[ni] = *reinterpret_cast<const bf16x8*>(&Bs[st][r * BK + swz(r, kc) * 8]);
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int r = wm * 64 + mi * 16 + (lane & 15);
        xf[mi] = *reinterpret_cast<const bf16x8*>(&As[st][r * BK + swz(r, kc) * 8]);
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = mfma16(wf[ni], xf[mi], acc[mi][ni]);
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<bf16x8*>(&As[st ^ 1][lds_off[i]]) = xr[i];
        *reinterpret_cast<bf16x8*>(&Bs[st ^ 1][lds_off[i]]) = wr[i];
      }
    }
    __syncthreads();
  }

  // ---- fused per-task LoRA expand ---------------------------------------
  if (a.lora.enabled) {
    const GemmLora& L = a.lora;
    const bf16* U = (const bf16*)L.U;
    const int wm0 = m0 + wm * 64;
    const int mlast = min(m0 + BM, a.M) - 1;
    const int t0 = L.row_task[m0], t1 = L.row_task[mlast];
    for (int t = t0; t <= t1; ++t) {
      const int r = min(L.rank[t], L.max_rank) & ~7;
      if (r <= 0) continue;
      const int s0 = L.seg_row[t], s1 = L.seg_row[t + 1];
      if (s1 <= wm0 || s0 >= wm0 + 64) continue;
      for (int kk = 0; kk < r; kk += 32) {
        const int kof = kk + 8 * (lane >> 4);
        const bool kin = kof < r;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          int slot, nrow, nlim;
          if (SWIGLU) {
            const int s = wn * 4 + ni;
            slot = s & 1;
            nrow = n0 + (s >> 1) * 16 + (lane & 15);
            nlim = a.N;
            if (n0 + (s >> 1) * 16 >= a.N) continue;
          } else {
            const int nb = n0 + wn * 64 + ni * 16;
            if (nb >= a.N) continue;
            slot = nb / L.slot_width;
            nrow = nb - slot * L.slot_width + (lane & 15);
            nlim = L.slot_width;
          }
          if (L.B[slot] == nullptr) continue;
          const bf16* Bt = (const bf16*)L.B[slot][t];
          bf16x8 wf = {};
          if (kin && nrow < nlim) wf = *reinterpret_cast<const bf16x8*>(Bt + (int64_t)nrow * r + kof);
#pragma unroll
          for (int mi = 0; mi < 4; ++mi) {
            const int m = wm0 + mi * 16 + (lane & 15);
            bf16x8 xf = {};
            if (m >= s0 && m < s1 && m < a.M)
              xf = *reinterpret_cast<const bf16x8*>(U + (int64_t)m * L.ldu + L.ucol[slot] + kof);
            acc[mi][ni] = mfma16(wf, xf, acc[mi][ni]);
          }
        }
      }
    }
  }

  // ---- epilogue -----------------------------------------------------------
  const bf16* bias = (const bf16*)a.bias;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int m = m0 + wm * 64 + mi * 16 + (lane & 15);
    if (m >= a.M) continue;
    if (SWIGLU) {
#pragma unroll
      for (int ni = 0; ni < 4; ni += 2) {
        const int s = wn * 4 + ni;
        const int j = n0 + (s >> 1) * 16 + 4 * (lane >> 4);
        if (j >= a.N) continue;
        bf16x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = (bf16)(silu_f(acc[mi][ni][r]) * acc[mi][ni + 1][r]);
        *reinterpret_cast<bf16x4*>((bf16*)a.out + (int64_t)m * a.ldo + j) = o;
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int n = n0 + wn * 64 + ni * 16 + 4 * (lane >> 4);
        if (n >= a.N) continue;
        f32x4 v = acc[mi][ni];
        if (bias) {
          const bf16x4 bb = *reinterpret_cast<const bf16x4*>(bias + n);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] += (float)bb[r];
        }
        if (EPI == EPI_RESID) {
          float4* dst = reinterpret_cast<float4*>((float*)a.out + (int64_t)m * a.ldo + n);
          float4 o = *dst;
          o.x += v[0]; o.y += v[1]; o.z += v[2]; o.w += v[3];
          *dst = o;
        } else {
          bf16x4 o;
#pragma unroll
          for (int r = 0; r < 4; ++r) o[r] = (bf16)(EPI == EPI_GELU ? gelu_erf(v[r]) : v[r]);
          *reinterpret_cast<bf16x4*>((bf16*)a.out + (int64_t)m * a.ldo + n) = o;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32: LDS-tiled FMA GEMM, 64x64 tile, 4x4 outputs per thread.
// ---------------------------------------------------------------------------
template <int EPI, bool SWIGLU>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  constexpr int TM = 64, TN = 64, TK = 16;
  __shared__ float Xs[TK][TM + 4];
  __shared__ float Ws[TK][TN + 4];
  __shared__ float W2s[SWIGLU ? TK : 1][TN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int n_tiles_n = (a.N + TN - 1) / TN;
  const int tn = blockIdx.x % n_tiles_n, tm = blockIdx.x / n_tiles_n;
  const int m0 = tm * TM, n0 = tn * TN;
  const float* X = (const float*)a.X;
  const float* W = (const float*)a.W;
  const float* W2 = (const float*)a.W2;
  const int lrow = tid >> 2, kq = (tid & 3) * 4;
  const int xm = min(m0 + lrow, a.M - 1), wn_ = min(n0 + lrow, a.N - 1);
  float acc[4][4] = {}, acc2[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += TK) {
    const float4 xv = *reinterpret_cast<const float4*>(X + (int64_t)xm * a.ldx + k0 + kq);
    const float4 wv = *reinterpret_cast<const float4*>(W + (int64_t)wn_ * a.K + k0 + kq);
    Xs[kq + 0][lrow] = xv.x; Xs[kq + 1][lrow] = xv.y; Xs[kq + 2][lrow] = xv.z; Xs[kq + 3][lrow] = xv.w;
    Ws[kq + 0][lrow] = wv.x; Ws[kq + 1][lrow] = wv.y; Ws[kq + 2][lrow] = wv.z; Ws[kq + 3][lrow] = wv.w;
    if (SWIGLU) {
      const float4 w2 = *reinterpret_cast<const float4*>(W2 + (int64_t)wn_ * a.K + k0 + kq);
      W2s[kq + 0][lrow] = w2.x; W2s[kq + 1][lrow] = w2.y; W2s[kq + 2][lrow] = w2.z; W2s[kq + 3][lrow] = w2.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      float xa[4], wb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) xa[i] = Xs[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wb[j] = Ws[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += xa[i] * wb[j];
      if (SWIGLU) {
#pragma unroll
        for (int j = 0; j < 4; ++j) wb[j] = W2s[k][tx * 4 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc2[i][j] += xa[i] * wb[j];
      }
    }
    __syncthreads();
  }

  if (a.lora.enabled) {
    const GemmLora& L = a.lora;
    const float* U = (const float*)L.U;
    const int mlast = min(m0 + TM, a.M) - 1;
    const int t0 = L.row_task[m0], t1 = L.row_task[mlast];
    for (int t = t0; t <= t1; ++t) {
      const int r = min(L.rank[t], L.max_rank) & ~7;
      if (r <= 0) continue;
      const int s0 = L.seg_row[t], s1 = L.seg_row[t + 1];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m < s0 || m >= s1 || m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + tx * 4 + j;
          if (n >= a.N) continue;
          const int slot = SWIGLU ? 0 : n / L.slot_width;
          const int nrow = SWIGLU ? n : n - slot * L.slot_width;
          if (L.B[slot] != nullptr) {
            const float* Bt = (const float*)L.B[slot][t];
            const float* u = U + (int64_t)m * L.ldu + L.ucol[slot];
            float s = 0.f;
            for (int q = 0; q < r; ++q) s += u[q] * Bt[(int64_t)nrow * r + q];
            acc[i][j] += s;
          }
          if (SWIGLU && L.B[1] != nullptr) {
            const float* Bt2 = (const float*)L.B[1][t];
            const float* u2 = U + (int64_t)m * L.ldu + L.ucol[1];
            float s2 = 0.f;
            for (int q = 0; q < r; ++q) s2 += u2[q] * Bt2[(int64_t)nrow * r + q];
            acc2[i][j] += s2;
          }
        }
      }
    }
  }

  const float* bias = (const float*)a.bias;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    const int n = n0 + tx * 4;
    if (m >= a.M || n >= a.N) continue;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = acc[i][j] + (bias ? bias[n + j] : 0.f);
      if (SWIGLU) v[j] = silu_f(acc[i][j]) * acc2[i][j];
      else if (EPI == EPI_GELU) v[j] = gelu_erf(v[j]);
    }
    float* dst = (float*)a.out + (int64_t)m * a.ldo + n;
    if (EPI == EPI_RESID) {
      float4 o = *reinterpret_cast<float4*>(dst);
      o.x += v[0]; o.y += v[1]; o.z += v[2]; o.w += v[3];
      *reinterpret_cast<float4*>(dst) = o;
    } else {
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

template <int EPI, bool SW>
hipError_t launch_one(int dtype, const GemmArgs& a, hipStream_t s) {
  if (dtype == VFM_BF16) {
    const int nt = SW ? BN / 2 : BN;
    const int grid = ((a.M + BM - 1) / BM) * ((a.N + nt - 1) / nt);
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI, SW>), dim3(grid), dim3(256), 0, s, a);
  } else {
    const int grid = ((a.M + 63) / 64) * ((a.N + 63) / 64);
    hipLaunchKernelGGL((gemm_f32_kernel<EPI, SW>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  switch (a.epi) {
    case EPI_STORE: return launch_one<EPI_STORE, false>(dtype, a, s);
    case EPI_GELU: return launch_one<EPI_GELU, false>(dtype, a, s);
    case EPI_RESID: return launch_one<EPI_RESID, false>(dtype, a, s);
    case EPI_SWIGLU: return launch_one<EPI_STORE, true>(dtype, a, s);
  }
  return hipErrorInvalidValue;
}
