// Attention per request (a6), RoPE (a5) and the KV-cache write.
//
// Attention never mixes requests: every kernel below maps a block to rows of
// ONE request (plan cu_seqlens), so co-batched tasks cannot influence each
// other (the isolation the paper's shared batch must keep, Section 3.1 R3).
//
// Prefill (bf16, MFMA): one block = 64 queries of one request and one head,
// 4 waves x 16 queries, online softmax over 64-key blocks staged in LDS.
// The score tile is computed transposed, S^T = K Q^T (K rows in the MFMA A
// slot, the wave's 16 queries in the B slot), so each lane holds 4 keys of
// ONE query; the max / sum reductions are in-lane plus two cross-lane
// shuffles, and exp(S^T) is already laid out as the B operand of
// O^T = V^T P^T (V is staged transposed in LDS).  Each lane finishes with 4
// consecutive head dims of one query: 8-byte stores.
//
// Decode (memory bound): one block per (request, head); 16 lane-groups of
// 16 lanes stream the request's cached keys, 16 bytes per lane per key row,
// each group with its own running max / sum / output, merged through LDS.
#include <algorithm>
#include <type_traits>

#include "vfm_internal.h"

namespace {

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

constexpr float LOG2E = 1.4426950408889634f;

// 2^x for the softmax, where x <= 0 after the max subtraction: the hardware
// v_exp_f32 directly (no range reduction needed; -inf gives 0).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// Sum over aligned groups of N lanes (N = 8 or 16) with DPP moves, which
// stay in the VALU: quad swaps, then the 8-lane and 16-lane mirrors pair
// each half with the other.
template <int N>
__device__ __forceinline__ float key_row_sum(float s) {
  static_assert(N == 8 || N == 16, "8 or 16 lanes per key row");
  auto dpp = [](float v, auto ctrl) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), decltype(ctrl)::value, 0xF, 0xF, true));
  };
  s += dpp(s, std::integral_constant<int, 0xB1>{});    // quad_perm [1, 0, 3, 2]
  s += dpp(s, std::integral_constant<int, 0x4E>{});    // quad_perm [2, 3, 0, 1]
  s += dpp(s, std::integral_constant<int, 0x141>{});   // row_half_mirror
  if constexpr (N == 16) s += dpp(s, std::integral_constant<int, 0x140>{});   // row_mirror
  return s;
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef bf16 bf16x2 __attribute__((ext_vector_type(2)));
// eight floats -> one bf16x8 MFMA operand with four packed conversions
__device__ __forceinline__ bf16x8 pack8(const f32x4& a, const f32x4& b) {
  const bf16x2 p0 = __builtin_convertvector(f32x2{a[0], a[1]}, bf16x2);
  const bf16x2 p1 = __builtin_convertvector(f32x2{a[2], a[3]}, bf16x2);
  const bf16x2 p2 = __builtin_convertvector(f32x2{b[0], b[1]}, bf16x2);
  const bf16x2 p3 = __builtin_convertvector(f32x2{b[2], b[3]}, bf16x2);
  const bf16x4 lo = __builtin_shufflevector(p0, p1, 0, 1, 2, 3);
  const bf16x4 hi = __builtin_shufflevector(p2, p3, 0, 1, 2, 3);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}
constexpr float NEG_BIG = -1e30f;

// ---------------------------------------------------------------------------
// RoPE, rotate-half: (x_i, x_{i+dh/2}) rotated by pos * theta^(-2i/dh).
// One block per row: the row's dh/2 angles (they do not depend on the head)
// go through LDS once, then each thread rotates 8 pairs of one head of q and
// of k with 16-byte accesses.  With a KV cache the same pass writes the
// rotated key and the value row to their cache slots (the cache-write kernel
// is then skipped).
// ---------------------------------------------------------------------------
// 8 consecutive elements (16-byte aligned for bf16, 32-byte for fp32) as floats
template <typename T>
__device__ inline void load8(const T* p, float (&v)[8]);
template <>
__device__ inline void load8<bf16>(const bf16* p, float (&v)[8]) {
  const bf16x8 x = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)x[i];
}
template <>
__device__ inline void load8<float>(const float* p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <typename T>
__device__ inline void store8(T* p, const float (&v)[8]);
template <>
__device__ inline void store8<bf16>(bf16* p, const float (&v)[8]) {
  bf16x8 x;
#pragma unroll
  for (int i = 0; i < 8; ++i) x[i] = (bf16)v[i];
  *reinterpret_cast<bf16x8*>(p) = x;
}
template <>
__device__ inline void store8<float>(float* p, const float (&v)[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(Plan pl, T* __restrict__ qkv, int d, int H, int dh,
                                                   float log2_theta, T* __restrict__ kc, T* __restrict__ vc,
                                                   int64_t kv_slots, KvPages kp) {
  __shared__ float cs_s[64], sn_s[64];        // dh / 2 <= 64
  const int r = blockIdx.x;
  const int half = dh >> 1;
  if (threadIdx.x < half) {
    const float inv = exp2f(-(2.0f * (float)threadIdx.x / (float)dh) * log2_theta);
    float sn, cs;
    sincosf((float)pl.pos[r] * inv, &sn, &cs);
    cs_s[threadIdx.x] = cs;
    sn_s[threadIdx.x] = sn;
  }
  __syncthreads();
  const int per_head = half / 8;              // 8-pair groups per head
  T* row = qkv + (int64_t)r * 3 * d;
  const int64_t slot = kc != nullptr ? kv_slot(pl, kp, pl.row_req[r], pl.pos[r]) : 0;
  for (int w = threadIdx.x; w < 2 * H * per_head; w += blockDim.x) {
    const int part = w / (H * per_head);      // q, then k
    const int hh = (w / per_head) % H;
    const int i0 = (w % per_head) * 8;
    T* x = row + part * d + hh * dh + i0;
    float a[8], b[8];
    load8<T>(x, a);
    load8<T>(x + half, b);
    float ya[8], yb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float c = cs_s[i0 + j], sv = sn_s[i0 + j];
      ya[j] = a[j] * c - b[j] * sv;
      yb[j] = a[j] * sv + b[j] * c;
    }
    store8<T>(x, ya);
    store8<T>(x + half, yb);
    if (kc != nullptr && part == 1) {         // the rotated key also goes to the cache
      T* kd = kc + ((int64_t)hh * kv_slots + slot) * dh + i0;
      store8<T>(kd, ya);
      store8<T>(kd + half, yb);
    }
  }
  if (kc != nullptr) {                        // and the value row, 8 elements per thread
    for (int c = 8 * threadIdx.x; c < d; c += 8 * blockDim.x) {
      const int hh = c / dh;
      float v[8];
      load8<T>(row + 2 * d + c, v);
      store8<T>(vc + ((int64_t)hh * kv_slots + slot) * dh + (c - hh * dh), v);
    }
  }
}

// ---------------------------------------------------------------------------
// KV-cache write: row r's k / v go to the slot of position pos[r] of its
// request (kv_start[p] + pos[r], or through the page table) in every head.
// The caches are head-major, [n_heads][kv_slots][head_dim], so one head's
// keys of one request (of one page, when paged) are a contiguous run.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void kv_write_kernel(Plan pl, const T* __restrict__ qkv, int d, int dh,
                                                       int64_t kv_slots, KvPages kp, T* __restrict__ kc,
                                                       T* __restrict__ vc) {
  const int r = blockIdx.x;
  const int p = pl.row_req[r];
  const int64_t slot = kv_slot(pl, kp, p, pl.pos[r]);
  const T* src = qkv + (int64_t)r * 3 * d;
  for (int c = 8 * threadIdx.x; c < d; c += 8 * 256) {   // 8 elements (16 B bf16) per thread
    const int h = c / dh;
    const int64_t o = ((int64_t)h * kv_slots + slot) * dh + (c - h * dh);
    float kv8[8];
    load8<T>(src + d + c, kv8);
    store8<T>(kc + o, kv8);
    load8<T>(src + 2 * d + c, kv8);
    store8<T>(vc + o, kv8);
  }
}

// K is stored unpadded with an XOR chunk swizzle (16-byte chunk kc of key r
// at kc ^ ((r >> 1) & 7) for 128-byte rows, kc ^ (r & 15) for 256-byte rows),
// which makes the 16-row fragment reads bank-conflict free on gfx950.
template <int DH>
__device__ __forceinline__ int kswz(int r, int kc) {
  return DH == 64 ? (kc ^ ((r >> 1) & 7)) : (kc ^ (r & 15));
}

// Short-sequence kernel: score sub-tiles 2u and 2u+1 take the keys of the
// 32-key block u in the order that leaves each lane, after S^T = K Q^T, with
// 8 consecutive keys across the pair (row x of the even sub-tile is key
// 32u + 8(x >> 2) + (x & 3), of the odd one 4 keys further), so the P^T
// operand's keys are contiguous and each V^T fragment is one 16-byte read.
// The K rows' chunk swizzle is a bijection of the bits that differ among the
// 16 rows one fragment read touches (row & 3 and (row >> 3) & 3), so those
// reads stay bank-conflict free.
template <int DH>
__device__ __forceinline__ int sswz(int r, int kc) {
  return DH == 64 ? (kc ^ (((r >> 1) & 1) | (((r >> 3) & 3) << 1)))
                  : (kc ^ ((r & 3) | (((r >> 3) & 3) << 2)));
}
__device__ __forceinline__ int pair_key(int ks, int x) {  // key of row x of sub-tile ks
  return (ks >> 1) * 32 + 8 * (x >> 2) + (x & 3) + 4 * (ks & 1);
}

// ---------------------------------------------------------------------------
// Prefill attention, bf16, MFMA: one block = 64 queries of one request and
// one head, 4 waves x 16 queries, online softmax over 64-key blocks.  K and V
// of a key block are staged in LDS row-major, as loaded (rows swizzled); the
// next block's K / V are loaded into registers while the current one is
// computed.  Score sub-tiles take the keys of each 32-key pair in the
// pair_key order, so a lane's P^T keys are contiguous; the V^T operand of
// O^T = V^T P^T is read from the row-major V tile with gfx950's transposing
// LDS read (ds_read_b64_tr_b16, vtr_frag), so V is never transposed in
// registers.  Causal: a wave skips key blocks entirely past its queries and
// masks only the block on its diagonal.  The causal variant is built for 3
// waves per SIMD (168 VGPRs, no spills; 3 blocks of 32 KB LDS per CU) instead
// of the 2 its unconstrained 204 registers allow: the extra resident block
// hides the per-step staging and barriers of the others.
// ---------------------------------------------------------------------------
// V tile row-major in LDS ([64 keys][DH] bf16) with 32-byte segments
// swizzled per row: segment s of key row r sits at s ^ vswz(r).  vswz makes
// the transposing reads below bank-conflict free (each 32-lane half of a read
// touches 8 rows, one 32-byte segment each, spread over all 64 banks) and is
// a permutation within the row, so the row stores stay conflict-free too.
template <int DH>
__device__ __forceinline__ int vswz(int r) {
  return DH == 128 ? ((r & 3) | (((r >> 3) & 1) << 2)) : (((r >> 1) & 1) | (((r >> 3) & 1) << 1));
}
// physical 16-byte chunk of logical chunk ch (head dims 8 ch .. 8 ch + 7) of row r
template <int DH>
__device__ __forceinline__ int vswz_chunk(int r, int ch) {
  return (((ch >> 1) ^ vswz<DH>(r)) << 1) | (ch & 1);
}
// ds_read_b64_tr_b16 (gfx950): within each group of 16 lanes, lane k brings
// the 4 consecutive 16-bit values D_k at its address and lane i receives
// D_{4j + i/4}[i % 4] for j = 0..3 (its lane layout, checked on the device).
// The A operand of v_mfma_f32_16x16x32_bf16 for V^T (lane l: head dim
// 16 ds + l % 16, keys 8 (l / 16) .. + 7 of the 32-key half u) is then two
// such reads: lane l points at key row 32 u + 8 (l / 16) + (l % 16) / 4 + 4 h
// (h = 0, 1: keys 0..3 and 4..7), dims 16 ds + 4 (l % 4) .. + 3.  With the
// row swizzle above the lane's segment term, vswz of that row, depends on
// the lane only, so one base offset serves every (u, h, ds).
template <int DH>
__device__ __forceinline__ int vtr_lane_offset(int lane) {
  const int g = lane >> 4, kq = lane & 15;
  const int row = 8 * g + (kq >> 2);        // + 32 u + 4 h, which leave vswz unchanged
  return row * DH * 2 + (vswz<DH>(row) << 5) + (kq & 3) * 8;
}
typedef short s16x4 __attribute__((ext_vector_type(4)));
template <int DH>
__device__ __forceinline__ bf16x8 vtr_frag(const bf16* Vs, int vbase, int u, int ds) {
  const char* p = reinterpret_cast<const char*>(Vs) + (vbase ^ (ds << 5)) + u * 32 * DH * 2;
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * DH * 2));
  bf16x8 f;
  __builtin_memcpy(&f, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&f) + 8, &hi, 8);
  return f;
}

template <int DH, bool CAUSAL, bool FROM_CACHE = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(CAUSAL ? 3 : 2))) void attn_prefill_bf16_kernel(Plan pl, const bf16* __restrict__ qkv,
                                                                int d, bf16* __restrict__ out,
                                                                float scale_log2, int skip_len,
                                                                const bf16* __restrict__ kc = nullptr,
                                                                const bf16* __restrict__ vc = nullptr,
                                                                int64_t kv_slots = 0, KvPages kpg = {}) {
  constexpr int KB = 64;          // keys per block step
  constexpr int CH = DH / 8;      // 16-byte chunks per key row
  constexpr int KPT = KB * CH / 256;          // K (and V) chunks per thread
  __shared__ __attribute__((aligned(16))) bf16 Ks[KB * DH];
  __shared__ __attribute__((aligned(16))) bf16 Vs[KB * DH];
  const int b = blockIdx.x, h = blockIdx.y;
  const int p = upper_index(pl.qblk_off, pl.n_req + 1, b);
  const int R = pl.cu_seqlens[p];
  const int L = pl.cu_seqlens[p + 1] - R;
  // FROM_CACHE (a prompt chunk after ctx cached tokens): every key, the
  // cached ones and the chunk's own, is read from the cache, where the RoPE
  // pass has already put the chunk's rows; query i sits at position ctx + i
  const int ctx = FROM_CACHE ? pl.ctx[p] : 0;
  if (FROM_CACHE && (ctx == 0 || L == 1)) return;   // block-uniform: other kernels' requests
  if (!FROM_CACHE && L <= skip_len) return;        // the whole-request kernel's
  const int NK = ctx + L;                          // keys of the request
  const int q0 = (b - pl.qblk_off[p]) * 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4;
  const int qi = q0 + wave * 16 + (lane & 15);  // this lane's query (B-operand column)
  const int64_t ld = 3 * (int64_t)d;
  const bf16* base = qkv + (int64_t)R * ld + h * DH;

  bf16x8 qf[DH / 32];
  {
    const bf16* qrow = base + (int64_t)min(qi, L - 1) * ld + 8 * g;
#pragma unroll
    for (int s2 = 0; s2 < DH / 32; ++s2) qf[s2] = *reinterpret_cast<const bf16x8*>(qrow + s2 * 32);
  }
  f32x4 o[DH / 16];
#pragma unroll
  for (int i = 0; i < DH / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = NEG_BIG, l_run = 0.f;

  // staging registers of one key block
  bf16x8 kr[KPT], vr[KPT];
  // where key k's K / V row of this head starts
  auto krow = [&](int k) -> const bf16* {
    if (FROM_CACHE) return kc + ((int64_t)h * kv_slots + kv_slot(pl, kpg, p, k)) * DH;
    return base + (int64_t)k * ld + d;
  };
  auto vrow = [&](int k) -> const bf16* {
    if (FROM_CACHE) return vc + ((int64_t)h * kv_slots + kv_slot(pl, kpg, p, k)) * DH;
    return base + (int64_t)k * ld + 2 * d;
  };
  auto load = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i, key = c / CH, ch = c % CH;
      kr[i] = bf16x8{};
      if (kb + key < NK) kr[i] = *reinterpret_cast<const bf16x8*>(krow(kb + key) + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i, key = c / CH, ch = c % CH;
      vr[i] = bf16x8{};
      if (kb + key < NK) vr[i] = *reinterpret_cast<const bf16x8*>(vrow(kb + key) + ch * 8);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i, key = c / CH, ch = c % CH;
      *reinterpret_cast<bf16x8*>(&Ks[key * DH + sswz<DH>(key, ch) * 8]) = kr[i];
    }
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + 256 * i, key = c / CH, ch = c % CH;
      *reinterpret_cast<bf16x8*>(&Vs[key * DH + vswz_chunk<DH>(key, ch) * 8]) = vr[i];
    }
  };

  const int kend = CAUSAL ? min(NK, ctx + q0 + 64) : NK;
  const int x = lane & 15;
  const int ke = pair_key(0, x), ko = pair_key(1, x);
  int koff_e = ke * DH, koff_o = ko * DH;
  const int vbase = vtr_lane_offset<DH>(lane);  // bytes, key row 8g + (x >> 2) of the tile
  asm volatile("" : "+v"(koff_e), "+v"(koff_o));
  const int wq0 = ctx + q0 + wave * 16;           // the wave's first query position
  int lim = CAUSAL ? min(NK, ctx + qi + 1) : NK;  // keys >= lim are masked for this lane

  load(0);
  store();
  __syncthreads();
  for (int kb = 0; kb < kend; kb += KB) {
    const bool more = kb + KB < kend;
    if (more) load(kb + KB);                      // in flight during this block's compute
    // keys of this block past the wave's last query (causal) or past L are all masked
    if (!CAUSAL || kb <= wq0 + 15) {
      f32x4 st[4];
      float mb = NEG_BIG;
      const bool full = kb + KB <= NK && (!CAUSAL || kb + KB <= wq0 + 1);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int row0 = (ks & 1) ? ko : ke;
        const bf16* kp = Ks + ((ks & 1) ? koff_o : koff_e) + (ks >> 1) * 32 * DH;
        f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s2 = 0; s2 < DH / 32; ++s2) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kp + sswz<DH>(row0, s2 * 4 + g) * 8);
          a = mfma16(kf, qf[s2], a);
        }
        if (!full) {
#pragma unroll
          for (int i = 0; i < 4; ++i) a[i] = kb + pair_key(ks, 4 * g + i) >= lim ? -INFINITY : a[i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) mb = fmaxf(mb, a[i]);
        st[ks] = a;
      }
      mb = fmaxf(mb, __shfl_xor(mb, 16, 64));
      mb = fmaxf(mb, __shfl_xor(mb, 32, 64));
      const float m_new = fmaxf(m_run, mb * scale_log2);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      float lsum = 0.f;
#pragma unroll
      for (int i = 0; i < DH / 16; ++i) o[i] *= alpha;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        f32x4 e0, e1;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          e0[i] = fast_exp2(fmaf(st[2 * u][i], scale_log2, -m_new));
          e1[i] = fast_exp2(fmaf(st[2 * u + 1][i], scale_log2, -m_new));
          lsum += e0[i] + e1[i];
        }
        const bf16x8 pf = pack8(e0, e1);
#pragma unroll
        for (int ds = 0; ds < DH / 16; ++ds) {
          const bf16x8 vf = vtr_frag<DH>(Vs, vbase, u, ds);
          o[ds] = mfma16(vf, pf, o[ds]);
        }
      }
      l_run = l_run * alpha + lsum;
    }
    __syncthreads();                              // every wave is done with this block's K / V^T
    if (more) {
      store();
      __syncthreads();
    }
  }
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (qi < L) {
    const float inv = 1.f / l_run;
    bf16* orow = out + (int64_t)(R + qi) * d + h * DH + 4 * g;
#pragma unroll
    for (int ds = 0; ds < DH / 16; ++ds) {
      bf16x4 v;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = (bf16)(o[ds][i] * inv);
      *reinterpret_cast<bf16x4*>(orow + ds * 16) = v;
    }
  }
}


// ---------------------------------------------------------------------------
// Prefill attention for requests of at most 256 tokens (bf16, MFMA, head
// dim 64; the launcher picks it by each request's own length).  NW waves
// take the 16-query groups in turn: with 8 (the launcher's choice) a
// 197-token request's 13 groups cost a wave at most 2 instead of 4, and two
// such blocks (56 KB of LDS, 124 VGPRs) still share a CU.
// One block per (request, head): K and V of the whole request are staged in
// LDS once, row-major (V^T fragments come from the transposing LDS read, as
// in the flash kernel), then each wave takes 16-query groups; with all keys
// resident the softmax is one pass (max, exp, sum) with no rescaling.  Keys
// are padded to a multiple of 32 with zeros and masked.
// ---------------------------------------------------------------------------
template <int DH, bool CAUSAL, int NKS, int NW = 4>
__global__ __launch_bounds__(64 * NW) void attn_short_bf16_kernel(Plan pl, const bf16* __restrict__ qkv,
                                                              int d, bf16* __restrict__ out,
                                                              float scale_log2) {
  // NKS 16-key sub-tiles cover every request of the batch (NKS * 16 >= L)
  constexpr int LMAX = NKS * 16;
  constexpr int CH = DH / 8;      // 16-byte chunks per key row
  __shared__ __attribute__((aligned(16))) bf16 Ks[LMAX * DH];
  __shared__ __attribute__((aligned(16))) bf16 Vs[LMAX * DH];
  const int p = blockIdx.x, h = blockIdx.y;
  const int R = pl.cu_seqlens[p];
  const int L = pl.cu_seqlens[p + 1] - R;
  if (L > LMAX) return;                         // block-uniform: a flash-kernel request
  constexpr int Lp = LMAX;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int64_t ld = 3 * (int64_t)d;
  const bf16* base = qkv + (int64_t)R * ld + h * DH;

  // Stage K and V.  Every global load of a thread is issued before its
  // first LDS store, so the block pays the load latency once.
  {
    constexpr int NT = 64 * NW;
    constexpr int KPT = (LMAX * CH + NT - 1) / NT;  // K (and V) chunks per thread
    bf16x8 kr[KPT], vr[KPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + NT * i, key = c / CH, ch = c % CH;
      kr[i] = bf16x8{};
      vr[i] = bf16x8{};
      if (key < L && c < LMAX * CH) {
        kr[i] = *reinterpret_cast<const bf16x8*>(base + (int64_t)key * ld + d + ch * 8);
        vr[i] = *reinterpret_cast<const bf16x8*>(base + (int64_t)key * ld + 2 * d + ch * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int c = tid + NT * i, key = c / CH, ch = c % CH;
      if (c < LMAX * CH) {
        *reinterpret_cast<bf16x8*>(&Ks[key * DH + sswz<DH>(key, ch) * 8]) = kr[i];
        *reinterpret_cast<bf16x8*>(&Vs[key * DH + vswz_chunk<DH>(key, ch) * 8]) = vr[i];
      }
    }
  }
  __syncthreads();

  auto load_q = [&](int qg, bf16x8 (&qf)[DH / 32]) {
    const int qi = qg * 16 + (lane & 15);
    const bf16* qrow = base + (int64_t)min(qi, L - 1) * ld + 8 * g;
#pragma unroll
    for (int s2 = 0; s2 < DH / 32; ++s2) qf[s2] = *reinterpret_cast<const bf16x8*>(qrow + s2 * 32);
  };
  bf16x8 qnext[DH / 32];
  if (wave * 16 < L) load_q(wave, qnext);
  for (int qg = wave; qg * 16 < L; qg += NW) {
    const int qi = qg * 16 + (lane & 15);
    bf16x8 qf[DH / 32];
#pragma unroll
    for (int s2 = 0; s2 < DH / 32; ++s2) qf[s2] = qnext[s2];
    if ((qg + NW) * 16 < L) load_q(qg + NW, qnext);   // in flight during this group
    f32x4 st[NKS];
    float mx = NEG_BIG;
    // The key swizzle of row 16*ks + (lane & 15) does not depend on ks, so
    // every fragment address is a per-lane base plus a constant offset.
    // keep the fragment reads inside this loop: hoisting all of them out
    // (they do not depend on the query group) needs ~2x the registers.  The
    // offset, not the pointer, goes through the empty asm, so the compiler
    // still knows the reads are LDS reads (ds_read, not flat loads).
    int koff = (lane & 15) * DH;
    asm volatile("" : "+v"(koff));
    const bf16* kbase = Ks + koff;
    // Scores stay unscaled here (the scale is positive, so the max commutes
    // with it); only key pairs that can hold a masked key pay for the mask:
    // the padded tail past L, and for causal rows the pairs that reach past
    // the group's first query.  Lane (x = lane & 15, g) of sub-tile ks holds
    // keys pair_key(ks, 4g + i), i < 4, of query x.
    const int x = lane & 15;
    const int ke = pair_key(0, x), ko = pair_key(1, x);   // rows of the even / odd sub-tile of pair 0
    // key pairs below nfull hold no masked key for any query of the group;
    // in the others, keys >= lim are masked for this lane's query (lim is
    // made opaque per group so the compares are not hoisted out of the loop
    // as dozens of lane masks held in scalar registers)
    const int nfull = (CAUSAL ? min(L, qg * 16 + 1) : L) >> 5;
    int lim = CAUSAL ? min(L, qi + 1) : L;
    asm volatile("" : "+v"(lim));
    int koff_e = ke * DH, koff_o = ko * DH;
    asm volatile("" : "+v"(koff_e), "+v"(koff_o));
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int row0 = (ks & 1) ? ko : ke;
      const bf16* kb = Ks + ((ks & 1) ? koff_o : koff_e) + (ks >> 1) * 32 * DH;
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s2 = 0; s2 < DH / 32; ++s2) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kb + sswz<DH>(row0, s2 * 4 + g) * 8);
        a = mfma16(kf, qf[s2], a);
      }
      if ((ks >> 1) < nfull) {
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, a[i]);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          a[i] = pair_key(ks, 4 * g + i) >= lim ? -INFINITY : a[i];
          mx = fmaxf(mx, a[i]);
        }
      }
      st[ks] = a;
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mxs = -mx * scale_log2;   // exp2(s * scale - max * scale), one fma per score
    float lsum = 0.f;
    f32x4 o[DH / 16];
#pragma unroll
    for (int i = 0; i < DH / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    int vbase = vtr_lane_offset<DH>(lane);
    asm volatile("" : "+v"(vbase));
#pragma unroll
    for (int u = 0; u < NKS / 2; ++u) {
      f32x4 e0, e1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e0[i] = fast_exp2(fmaf(st[2 * u][i], scale_log2, mxs));
        e1[i] = fast_exp2(fmaf(st[2 * u + 1][i], scale_log2, mxs));
        lsum += e0[i] + e1[i];
      }
      const bf16x8 pf = pack8(e0, e1);
#pragma unroll
      for (int ds = 0; ds < DH / 16; ++ds) {
        const bf16x8 vf = vtr_frag<DH>(Vs, vbase, u, ds);
        o[ds] = mfma16(vf, pf, o[ds]);
      }
    }
    lsum += __shfl_xor(lsum, 16, 64);
    lsum += __shfl_xor(lsum, 32, 64);
    if (qi < L) {
      const float inv = 1.f / lsum;
      bf16* orow = out + (int64_t)(R + qi) * d + h * DH + 4 * g;
#pragma unroll
      for (int ds = 0; ds < DH / 16; ++ds) {
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = (bf16)(o[ds][i] * inv);
        *reinterpret_cast<bf16x4*>(orow + ds * 16) = v;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Prefill attention, generic SIMT (fp32 workloads): 64 queries per block,
// 4 threads per query, each owning DH/4 dims; keys staged in LDS.
// ---------------------------------------------------------------------------
template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_prefill_simt_kernel(Plan pl, const T* __restrict__ qkv,
                                                                int d, T* __restrict__ out,
                                                                float scale_log2, int causal) {
  constexpr int DQ = DH / 4;
  __shared__ float Ks[64][DH + 1];
  __shared__ float Vs[64][DH + 1];
  const int b = blockIdx.x, h = blockIdx.y;
  const int p = upper_index(pl.qblk_off, pl.n_req + 1, b);
  const int R = pl.cu_seqlens[p];
  const int L = pl.cu_seqlens[p + 1] - R;
  const int q0 = (b - pl.qblk_off[p]) * 64;
  const int tid = threadIdx.x, qi = q0 + (tid >> 2), part = tid & 3;
  const int64_t ld = 3 * (int64_t)d;
  float q[DQ], o[DQ];
  const T* qrow = qkv + (int64_t)(R + min(qi, L - 1)) * ld + h * DH + part * DQ;
#pragma unroll
  for (int i = 0; i < DQ; ++i) { q[i] = to_f32(qrow[i]); o[i] = 0.f; }
  float m_run = NEG_BIG, l_run = 0.f;
  const int kend = causal ? min(L, q0 + 64) : L;
  for (int kb = 0; kb < kend; kb += 64) {
    for (int e = tid; e < 64 * DH; e += 256) {
      const int key = e / DH, c = e % DH;
      float kv = 0.f, vv = 0.f;
      if (kb + key < L) {
        const T* src = qkv + (int64_t)(R + kb + key) * ld + h * DH + c;
        kv = to_f32(src[d]);
        vv = to_f32(src[2 * d]);
      }
      Ks[key][c] = kv;
      Vs[key][c] = vv;
    }
    __syncthreads();
    const int nk = min(64, kend - kb);
    for (int j = 0; j < nk; ++j) {
      const int key = kb + j;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < DQ; ++i) s += q[i] * Ks[j][part * DQ + i];
      s += __shfl_xor(s, 1, 64);
      s += __shfl_xor(s, 2, 64);
      s *= scale_log2;
      if (causal && key > qi) continue;
      const float m_new = fmaxf(m_run, s);
      const float alpha = exp2f(m_run - m_new), e = exp2f(s - m_new);
      l_run = l_run * alpha + e;
#pragma unroll
      for (int i = 0; i < DQ; ++i) o[i] = o[i] * alpha + e * Vs[j][part * DQ + i];
      m_run = m_new;
    }
    __syncthreads();
  }
  if (qi < L) {
    T* orow = out + (int64_t)(R + qi) * d + h * DH + part * DQ;
#pragma unroll
    for (int i = 0; i < DQ; ++i) orow[i] = from_f32<T>(o[i] / l_run);
  }
}

// ---------------------------------------------------------------------------
// Decode attention: one query row per request against its cached keys
// (slots kv_start .. kv_start + ctx, the last one just written).
// ---------------------------------------------------------------------------

// The keys of a request are cut into DEC_CHUNK-key chunks, one block per
// (request, head, chunk), so long contexts spread over many CUs instead of
// finishing as a long tail; each block leaves its chunk's running max m,
// sum l and unnormalised output o, and a merge kernel combines the chunks
// (the usual rescaling of partial softmax sums by 2^(m_c - m)).  A request
// with a single chunk gets its output from the attention kernel directly.
// Inside a block, each group of LPK lanes walks one key stream; every step
// issues the K and V loads of UNR keys of the stream before any is used.
// PAGED: the request's keys sit in pages (KvPages); the block first reads
// its chunk's page ids (at most DEC_CHUNK / 16) into LDS.  mixed: prompts
// (ctx 0) of a continuous-batching step are left to the prefill kernels.
// 2048-key chunks: a request of up to 2048 cached keys is one block and
// needs no merge; against 1024-key chunks the 7B decode attention took 727
// instead of 766 us per layer (contexts of 256 to 2048 keys).
constexpr int DEC_CHUNK = 2048;

// In a mixed step, the requests the decode kernels own: one new row after
// cached tokens.
__device__ __forceinline__ bool decode_row(const Plan& pl, int p) {
  return pl.ctx[p] > 0 && pl.cu_seqlens[p + 1] - pl.cu_seqlens[p] == 1;
}
constexpr int DEC_MAX_PAGES = DEC_CHUNK / 16;   // page ids per chunk (pages of >= 16 slots)

// The chunk [kbeg, kend)'s page ids into spg; returns the first page index.
__device__ __forceinline__ int load_chunk_pages(const Plan& pl, const KvPages& kp, int p, int kbeg, int kend,
                                                int* spg) {
  const int first = kbeg >> kp.log2_page;
  const int npg = ((kend - 1) >> kp.log2_page) - first + 1;
  if ((int)threadIdx.x < npg)
    spg[threadIdx.x] = kp.table[(int64_t)pl.order[p] * kp.max_pages + first + threadIdx.x];
  __syncthreads();
  return first;
}

template <typename T, int DH, int UNR, bool PAGED>
__global__ __launch_bounds__(256) void attn_decode_kernel(Plan pl, const T* __restrict__ qkv, int d,
                                                          const T* __restrict__ kc,
                                                          const T* __restrict__ vc, int64_t kv_slots,
                                                          KvPages kpg, int mixed,
                                                          float* __restrict__ part, int nchunk,
                                                          float scale_log2, T* __restrict__ out) {
  using OT = T;
  constexpr int LPK = DH / 8;          // lanes per key row (8 dims each)
  constexpr int NG = 256 / LPK;        // key streams per block
  __shared__ float sm[NG], sl[NG];
  __shared__ float so[NG][DH + 1];
  __shared__ int spg[PAGED ? DEC_MAX_PAGES : 1];
  const int h = blockIdx.x, p = blockIdx.y, c = blockIdx.z;
  const int tid = threadIdx.x;
  const int grp = tid / LPK, sub = tid % LPK;
  if (mixed && !decode_row(pl, p)) return;   // a prompt or prompt chunk: block-uniform
  const int R = pl.cu_seqlens[p];            // the request's (single) query row
  const int nkeys = pl.ctx[p] + (pl.cu_seqlens[p + 1] - R);
  const int kbeg = c * DEC_CHUNK;
  if (kbeg >= nkeys) return;                 // block-uniform
  const int kend = min(kbeg + DEC_CHUNK, nkeys);
  const int pg0 = PAGED ? load_chunk_pages(pl, kpg, p, kbeg, kend, spg) : 0;
  const int64_t base = PAGED ? 0 : (int64_t)pl.kv_start[p];
  // element offset of key k of the request from the head's first slot
  auto koff = [&](int k) -> int64_t {
    if (!PAGED) return (int64_t)k * DH;
    const int lp = kpg.log2_page;
    return (((int64_t)spg[(k >> lp) - pg0] << lp) + (k & ((1 << lp) - 1))) * DH;
  };
  float q[8];
  load8<T>(qkv + (int64_t)R * 3 * d + h * DH + sub * 8, q);
  float m_run = NEG_BIG, l_run = 0.f, o[8] = {};
  const T* kp = kc + ((int64_t)h * kv_slots + base) * DH + sub * 8;
  const T* vp = vc + ((int64_t)h * kv_slots + base) * DH + sub * 8;
  for (int k0 = kbeg + grp; k0 < kend; k0 += UNR * NG) {
    float kv[UNR][8], vv[UNR][8];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int k = min(k0 + u * NG, kend - 1);   // clamped: masked below
      load8<T>(kp + koff(k), kv[u]);
      load8<T>(vp + koff(k), vv[u]);
    }
    float sc[UNR];
    float smax = NEG_BIG;
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) s += q[i] * kv[u][i];
      s = key_row_sum<LPK>(s);
      sc[u] = k0 + u * NG < kend ? s * scale_log2 : NEG_BIG;
      smax = fmaxf(smax, sc[u]);
    }
    const float m_new = fmaxf(m_run, smax);
    const float alpha = exp2f(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] *= alpha;
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const float e = k0 + u * NG < kend ? exp2f(sc[u] - m_new) : 0.f;
      l_run += e;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] += e * vv[u][i];
    }
    m_run = m_new;
  }
  if (sub == 0) { sm[grp] = m_run; sl[grp] = l_run; }
#pragma unroll
  for (int i = 0; i < 8; ++i) so[grp][sub * 8 + i] = o[i];
  __syncthreads();
  if (tid < DH) {
    float M = NEG_BIG;
    for (int gq = 0; gq < NG; ++gq) M = fmaxf(M, sm[gq]);
    float lsum = 0.f, acc = 0.f;
    for (int gq = 0; gq < NG; ++gq) {
      const float w = exp2f(sm[gq] - M);
      lsum += sl[gq] * w;
      acc += so[gq][tid] * w;
    }
    // partial record of (p, h, c): [m, l, o[0..DH)]
    if (nkeys <= DEC_CHUNK) {
      // the request's only chunk: its output directly (the merge skips it)
      out[(int64_t)R * d + h * DH + tid] = from_f32<OT>(acc / lsum);
    } else {
      float* rec = part + (((int64_t)p * gridDim.x + h) * nchunk + c) * (DH + 2);
      rec[2 + tid] = acc;
      if (tid == 0) { rec[0] = M; rec[1] = lsum; }
    }
  }
}

// bf16 variant with the next step's K / V loads in flight while the current
// step is computed: a two-slot register ring filled by loads the compiler
// does not track (so it does not wait for every load at the loop back-edge);
// the kernel's own waits cover them, as loads complete in issue order.  The
// loads carry the nontemporal hint: each cached key is read once per step,
// and a probe of this access pattern streams at 7.1 TB/s with the hint
// against 6.3 TB/s without it.
typedef bf16 bf16x2 __attribute__((ext_vector_type(2)));
// a0 * b0 + a1 * b1 + c on bf16 pairs, fp32 accumulation
__device__ __forceinline__ float dot2_bf16(bf16x2 a, bf16x2 b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(a, b, c, false);
}
__device__ __forceinline__ bf16x2 pair(const bf16x8& v, int j) { return bf16x2{v[2 * j], v[2 * j + 1]}; }

__device__ __forceinline__ void gload16_untracked(bf16x8& dst, const bf16* p) {
  asm volatile("global_load_dwordx4 %0, %1, off nt" : "=v"(dst) : "v"(p) : "memory");
}

template <int DH, int UNR, bool PAGED>
__global__ __launch_bounds__(256) void attn_decode_bf16_kernel(Plan pl, const bf16* __restrict__ qkv, int d,
                                                               const bf16* __restrict__ kc,
                                                               const bf16* __restrict__ vc, int64_t kv_slots,
                                                               KvPages kpg, int mixed,
                                                               float* __restrict__ part, int nchunk,
                                                               float scale_log2, bf16* __restrict__ out) {
  using OT = bf16;
  constexpr int LPK = DH / 8;          // lanes per key row (8 dims each)
  constexpr int NG = 256 / LPK;        // key streams per block
  constexpr int STEP = UNR * NG;       // keys per step of the block
  static_assert(UNR % 2 == 0, "keys are weighted in pairs");
  __shared__ float sm[NG], sl[NG];
  __shared__ float so[NG][DH + 1];
  __shared__ int spg[PAGED ? DEC_MAX_PAGES : 1];
  const int h = blockIdx.x, p = blockIdx.y, c = blockIdx.z;
  const int tid = threadIdx.x;
  const int grp = tid / LPK, sub = tid % LPK;
  if (mixed && !decode_row(pl, p)) return;   // a prompt or prompt chunk: block-uniform
  const int R = pl.cu_seqlens[p];
  const int nkeys = pl.ctx[p] + (pl.cu_seqlens[p + 1] - R);
  const int kbeg = c * DEC_CHUNK;
  if (kbeg >= nkeys) return;                 // block-uniform
  const int kend = min(kbeg + DEC_CHUNK, nkeys);
  const int pg0 = PAGED ? load_chunk_pages(pl, kpg, p, kbeg, kend, spg) : 0;
  const int64_t base = PAGED ? 0 : (int64_t)pl.kv_start[p];
  auto koff = [&](int k) -> int64_t {
    if (!PAGED) return (int64_t)k * DH;
    const int lp = kpg.log2_page;
    return (((int64_t)spg[(k >> lp) - pg0] << lp) + (k & ((1 << lp) - 1))) * DH;
  };
  const bf16x8 q = *reinterpret_cast<const bf16x8*>(qkv + (int64_t)R * 3 * d + h * DH + sub * 8);
  float m_run = NEG_BIG, l_run = 0.f, o[8] = {};
  const bf16* kp = kc + ((int64_t)h * kv_slots + base) * DH + sub * 8;
  const bf16* vp = vc + ((int64_t)h * kv_slots + base) * DH + sub * 8;
  bf16x8 kb[2][UNR], vb[2][UNR];
  // keys past the chunk re-read its last key (masked), so every step issues
  // 2 * UNR loads and one wait count holds throughout
  auto issue = [&](int slot, int k0) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int k = min(k0 + u * NG, kend - 1);
      gload16_untracked(kb[slot][u], kp + koff(k));
      gload16_untracked(vb[slot][u], vp + koff(k));
    }
  };
  auto step = [&](int slot, int k0) {
    float sc[UNR];
    float smax = NEG_BIG;
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) s = dot2_bf16(pair(q, j), pair(kb[slot][u], j), s);
      s = key_row_sum<LPK>(s);
      sc[u] = k0 + u * NG < kend ? s * scale_log2 : NEG_BIG;
      smax = fmaxf(smax, sc[u]);
    }
    const float m_new = fmaxf(m_run, smax);
    const float alpha = fast_exp2(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] *= alpha;
    // weights rounded to bf16 (as the MFMA paths do); the sum l takes the
    // rounded values so the normalisation matches
#pragma unroll
    for (int u = 0; u < UNR; u += 2) {
      const float e0 = k0 + u * NG < kend ? fast_exp2(sc[u] - m_new) : 0.f;
      const float e1 = k0 + (u + 1) * NG < kend ? fast_exp2(sc[u + 1] - m_new) : 0.f;
      const bf16x2 ep = {(bf16)e0, (bf16)e1};
      l_run += (float)ep[0] + (float)ep[1];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        o[i] = dot2_bf16(ep, bf16x2{vb[slot][u][i], vb[slot][u + 1][i]}, o[i]);
    }
    m_run = m_new;
  };
  const int first = kbeg + grp;
  // q is needed by the first step: take its (tracked) load's wait here,
  // before the untracked K / V loads are in flight behind it
  asm volatile("" ::"v"(q));
  if (first < kend) {
    issue(0, first);
    for (int k0 = first; k0 < kend; k0 += 2 * STEP) {
      issue(1, k0 + STEP);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * UNR) : "memory");   // slot 0 has landed
#pragma unroll
      for (int u = 0; u < UNR; ++u) asm volatile("" : "+v"(kb[0][u]), "+v"(vb[0][u]));
      step(0, k0);
      if (k0 + STEP >= kend) break;
      issue(0, k0 + 2 * STEP);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * UNR) : "memory");   // slot 1 has landed
#pragma unroll
      for (int u = 0; u < UNR; ++u) asm volatile("" : "+v"(kb[1][u]), "+v"(vb[1][u]));
      step(1, k0 + STEP);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  if (sub == 0) { sm[grp] = m_run; sl[grp] = l_run; }
#pragma unroll
  for (int i = 0; i < 8; ++i) so[grp][sub * 8 + i] = o[i];
  __syncthreads();
  if (tid < DH) {
    float M = NEG_BIG;
    for (int gq = 0; gq < NG; ++gq) M = fmaxf(M, sm[gq]);
    float lsum = 0.f, acc = 0.f;
    for (int gq = 0; gq < NG; ++gq) {
      const float w = exp2f(sm[gq] - M);
      lsum += sl[gq] * w;
      acc += so[gq][tid] * w;
    }
    if (nkeys <= DEC_CHUNK) {
      // the request's only chunk: its output directly (the merge skips it)
      out[(int64_t)R * d + h * DH + tid] = from_f32<OT>(acc / lsum);
    } else {
      float* rec = part + (((int64_t)p * gridDim.x + h) * nchunk + c) * (DH + 2);
      rec[2 + tid] = acc;
      if (tid == 0) { rec[0] = M; rec[1] = lsum; }
    }
  }
}

template <typename T, int DH>
__global__ __launch_bounds__(DH) void attn_decode_merge_kernel(Plan pl, const float* __restrict__ part,
                                                               int nchunk, int d, int mixed, T* __restrict__ out) {
  constexpr int MAXC = 64;                   // chunks merged per pass through LDS
  __shared__ float sw[MAXC];
  const int p = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  if (mixed && !decode_row(pl, p)) return;   // a prompt or prompt chunk (prefill kernels)
  const int R = pl.cu_seqlens[p];
  const int nkeys = pl.ctx[p] + (pl.cu_seqlens[p + 1] - R);
  const int nc = min((nkeys + DEC_CHUNK - 1) / DEC_CHUNK, nchunk);
  if (nc <= 1) return;                       // written by the attention kernel itself
  const float* rec = part + ((int64_t)p * gridDim.y + h) * nchunk * (DH + 2);
  // global max of the chunk maxima (all threads read the same few values)
  float M = NEG_BIG;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, rec[c * (DH + 2)]);
  float lsum = 0.f, acc = 0.f;
  for (int c0 = 0; c0 < nc; c0 += MAXC) {
    const int cn = min(MAXC, nc - c0);
    __syncthreads();
    if (tid < cn) sw[tid] = exp2f(rec[(c0 + tid) * (DH + 2)] - M);   // chunk weights, in parallel
    __syncthreads();
    int c = 0;
    for (; c + 4 <= cn; c += 4) {
      float o4[4], l4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        o4[j] = rec[(c0 + c + j) * (DH + 2) + 2 + tid];
        l4[j] = rec[(c0 + c + j) * (DH + 2) + 1];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        lsum += l4[j] * sw[c + j];
        acc += o4[j] * sw[c + j];
      }
    }
    for (; c < cn; ++c) {
      lsum += rec[(c0 + c) * (DH + 2) + 1] * sw[c];
      acc += rec[(c0 + c) * (DH + 2) + 2 + tid] * sw[c];
    }
  }
  out[(int64_t)R * d + h * DH + tid] = from_f32<T>(acc / lsum);
}

}  // namespace

hipError_t launch_rope(int dtype, const Plan& pl, void* qkv, int d, int n_heads, int head_dim,
                       float theta, void* k_cache, void* v_cache, int64_t kv_slots, const KvPages& kp,
                       hipStream_t s) {
  if (pl.T == 0) return hipSuccess;
  const float l2t = log2f(theta);
  if (dtype == VFM_BF16)
    hipLaunchKernelGGL(rope_kernel<bf16>, dim3(pl.T), dim3(256), 0, s, pl, (bf16*)qkv, d, n_heads, head_dim, l2t,
                       (bf16*)k_cache, (bf16*)v_cache, kv_slots, kp);
  else
    hipLaunchKernelGGL(rope_kernel<float>, dim3(pl.T), dim3(256), 0, s, pl, (float*)qkv, d, n_heads, head_dim, l2t,
                       (float*)k_cache, (float*)v_cache, kv_slots, kp);
  return hipGetLastError();
}

size_t attention_workspace(const vfm_cfg& c, const Plan& pl, int max_keys) {
  if (c.attn != VFM_ATTN_DECODE && c.attn != VFM_ATTN_MIXED) return 0;
  const int nchunk = (max_keys + DEC_CHUNK - 1) / DEC_CHUNK;
  return (size_t)pl.n_req * c.n_heads * nchunk * (c.head_dim + 2) * sizeof(float);
}

hipError_t launch_attention(int dtype, const Plan& pl, const vfm_cfg& c, const void* qkv, void* out,
                            void* k_cache, void* v_cache, int64_t kv_slots, const KvPages& kp, bool kv_written,
                            bool chunked, void* ws, size_t ws_bytes, int max_keys, hipStream_t s) {
  const int d = c.d_model, H = c.n_heads, DH = c.head_dim;
  const float scale_log2 = LOG2E / sqrtf((float)DH);
  const bool mixed = c.attn == VFM_ATTN_MIXED;
  // timing classes: the attention kernel itself is VFM_PROF_ATTN, the cache
  // write and the decode merge VFM_PROF_OTHER
  int pi = -1;
  if (k_cache && !kv_written && c.attn != VFM_ATTN_BIDIR) {
    pi = prof_begin(VFM_PROF_OTHER, s);
    if (dtype == VFM_BF16)
      hipLaunchKernelGGL(kv_write_kernel<bf16>, dim3(pl.T), dim3(256), 0, s, pl, (const bf16*)qkv, d, DH,
                         kv_slots, kp, (bf16*)k_cache, (bf16*)v_cache);
    else
      hipLaunchKernelGGL(kv_write_kernel<float>, dim3(pl.T), dim3(256), 0, s, pl, (const float*)qkv, d, DH,
                         kv_slots, kp, (float*)k_cache, (float*)v_cache);
    prof_end(pi, s);
  }
  // Prompts: causal (or bidirectional) attention over each request's own
  // rows.  In a mixed step this also covers the decode rows, each against
  // itself only; the decode kernels below overwrite those rows.
  if (c.attn != VFM_ATTN_DECODE) {
    pi = prof_begin(VFM_PROF_ATTN, s);
    dim3 grid(pl.n_qblocks, H);
    const bool causal = c.attn != VFM_ATTN_BIDIR;
    const int short_rows = DH == 64 ? VFM_SHORT_ATTN_ROWS : 0;   // whole-request kernel up to this
    if (dtype == VFM_BF16 && short_rows > 0 && pl.max_short > 0) {
      // requests of at most VFM_SHORT_ATTN_ROWS rows (the others return);
      // keys past a request's length add exact zeros, so the sub-tile count
      // does not change its result
      dim3 g2(pl.n_req, H);
      const int nks = ((pl.max_short + 31) / 32) * 2;   // 16-key sub-tiles, even
#define SHORT(D_, C_, N_)                                                                           \
  hipLaunchKernelGGL((attn_short_bf16_kernel<D_, C_, N_, 8>), g2, dim3(512), 0, s, pl, (const bf16*)qkv, \
                     d, (bf16*)out, scale_log2)
#define SHORT_N(D_, C_)                                            \
  switch (nks) {                                                   \
    case 2: SHORT(D_, C_, 2); break;   case 4: SHORT(D_, C_, 4); break;   \
    case 6: SHORT(D_, C_, 6); break;   case 8: SHORT(D_, C_, 8); break;   \
    case 10: SHORT(D_, C_, 10); break; case 12: SHORT(D_, C_, 12); break; \
    case 14: SHORT(D_, C_, 14); break; default: SHORT(D_, C_, 16); break; \
  }
      if (causal) { SHORT_N(64, true); } else { SHORT_N(64, false); }
#undef SHORT_N
#undef SHORT
    }
    if (dtype == VFM_BF16 && (short_rows == 0 || pl.n_long > 0)) {
      // requests longer than short_rows (the others return)
#define PRE(D_, C_)                                                                            \
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<D_, C_>), grid, dim3(256), 0, s, pl, (const bf16*)qkv, \
                     d, (bf16*)out, scale_log2, short_rows)
      if (DH == 64) { if (causal) PRE(64, true); else PRE(64, false); }
      else { if (causal) PRE(128, true); else PRE(128, false); }
#undef PRE
    }
    if (dtype != VFM_BF16) {
      if (DH == 64)
        hipLaunchKernelGGL((attn_prefill_simt_kernel<float, 64>), grid, dim3(256), 0, s, pl,
                           (const float*)qkv, d, (float*)out, scale_log2, (int)causal);
      else
        hipLaunchKernelGGL((attn_prefill_simt_kernel<float, 128>), grid, dim3(256), 0, s, pl,
                           (const float*)qkv, d, (float*)out, scale_log2, (int)causal);
    }
    // prompt chunks after cached tokens: their rows again, over every key
    // of the request read from the cache (the rows above attended to the
    // chunk alone)
    if (mixed && chunked && dtype == VFM_BF16) {
#define CHUNK(D_)                                                                                     \
  hipLaunchKernelGGL((attn_prefill_bf16_kernel<D_, true, true>), grid, dim3(256), 0, s, pl,           \
                     (const bf16*)qkv, d, (bf16*)out, scale_log2, 0, (const bf16*)k_cache,           \
                     (const bf16*)v_cache, kv_slots, kp)
      if (DH == 64) CHUNK(64); else CHUNK(128);
#undef CHUNK
    }
    prof_end(pi, s);
    if (!mixed) return hipGetLastError();
  }
  // Decode rows: one query against the request's cached keys.
  if (ws_bytes < attention_workspace(c, pl, max_keys)) return hipErrorInvalidValue;
  const int nchunk = (max_keys + DEC_CHUNK - 1) / DEC_CHUNK;
  float* part = (float*)ws;
  const int mx = mixed ? 1 : 0;
  dim3 grid(H, pl.n_req, nchunk), gm(pl.n_req, H);
  // 6 keys per key stream and step (7B decode layer, 2048-key chunks: 722 us
  // against 738 us with 4 and 731 us with 8, same machine)
#define DEC_K(PG, D_)                                                                                     \
  if (dtype == VFM_BF16)                                                                                   \
    hipLaunchKernelGGL((attn_decode_bf16_kernel<D_, 6, PG>), grid, dim3(256), 0, s, pl, (const bf16*)qkv, \
                       d, (const bf16*)k_cache, (const bf16*)v_cache, kv_slots, kp, mx, part, nchunk,   \
                       scale_log2, (bf16*)out);                                                          \
  else                                                                                                     \
    hipLaunchKernelGGL((attn_decode_kernel<float, D_, 4, PG>), grid, dim3(256), 0, s, pl,                 \
                       (const float*)qkv, d, (const float*)k_cache, (const float*)v_cache, kv_slots, kp, \
                       mx, part, nchunk, scale_log2, (float*)out)
#define DEC(TT, D_)                                                                                    \
  pi = prof_begin(VFM_PROF_ATTN, s);                                                                   \
  if (kp.table) { DEC_K(true, D_); } else { DEC_K(false, D_); }                                       \
  prof_end(pi, s);                                                                                     \
  if (nchunk > 1) { /* some request has more than one chunk to merge */                                \
    pi = prof_begin(VFM_PROF_OTHER, s);                                                                \
    hipLaunchKernelGGL((attn_decode_merge_kernel<TT, D_>), gm, dim3(D_), 0, s, pl, (const float*)part, \
                       nchunk, d, mx, (TT*)out);                                                       \
    prof_end(pi, s);                                                                                   \
  }
  if (dtype == VFM_BF16) {
    if (DH == 64) { DEC(bf16, 64); } else { DEC(bf16, 128); }
  } else {
    if (DH == 64) { DEC(float, 64); } else { DEC(float, 128); }
  }
#undef DEC
#undef DEC_K
  return hipGetLastError();
}
