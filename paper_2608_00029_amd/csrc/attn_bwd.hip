// Fused causal attention backward for gfx950: two kernels that recompute the
// probabilities from the forward's log-sum-exp (section 4.2, backward
// paragraph), so the S x S matrix never exists in memory, and that need no
// atomics (every output element is owned by exactly one workgroup, and its
// accumulation order is fixed, so results are bitwise reproducible).
//
//  dq kernel   (reduces over keys; one workgroup per 128 queries, 32 per wave)
//     D_i = sum_d dO_id O_id                      (float, written for the next kernel)
//     per 32-key block:  S^T = K Q^T,  dP^T = V dO^T          (matrix cores)
//                        P^T = exp2(S^T * scale*log2e - LSE_i*log2e)
//                        dS^T = P^T * (dP^T - D_i)
//                        dQ^T += K^T dS^T                      (matrix cores)
//     dQ = scale * dQ^T^T
//  dkdv kernel (reduces over queries; one workgroup per 128 keys, 32 per wave)
//     per 32-query block: S = Q K^T,  dP = dO V^T
//                         P = exp2(S * scale*log2e - LSE*log2e), dS = P * (dP - D)
//                         dV^T += dO^T P,  dK^T += Q^T dS
//     dK = scale * dK^T^T
//
// Both keep the score-like blocks in registers with one lane per query (dq)
// or per key (dkdv), so LSE and D are per-lane scalars in the dq kernel, and
// the probability block feeds the second contraction straight from registers.
// The causal triangle is exploited on both sides: the dq key loop stops at the
// diagonal (upper bound clamped), the dkdv query loop starts at it (lower bound
// raised), and only blocks straddling the diagonal or the ragged sequence end
// are masked.
#include "attn_device.h"
#include "attn_launch.h"

namespace cattn {

template <typename T, int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(const T* __restrict__ Q, const T* __restrict__ K,
                                                          const T* __restrict__ V, const T* __restrict__ O,
                                                          const T* __restrict__ dO, const float* __restrict__ LSE,
                                                          T* __restrict__ dQ, float* __restrict__ Dvec, int S,
                                                          int BH, int n_qtiles, float c, float scale, int H,
                                                          int seq_major) {
  typedef Mma<T> M;
  constexpr int BQ = 128, BK = 64, NT = 256;
  constexpr int KS_D = D / M::K, KS_32 = 32 / M::K, DT = D / 32;
  constexpr int TILE = BK * D * (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * TILE];  // [buffer][K, V]

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, qt;
  tile_of_block(blockIdx.x, BH, n_qtiles, CAUSAL, bh, qt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const T* Kb = K + base;
  const T* Vb = V + base;

  const int q0 = qt * BQ, qw = q0 + 32 * w, my_q = qw + r;
  typename M::frag qf[KS_D], dof[KS_D];
  load_row_frags<T, D>(Q + base, my_q, S, h, rs, qf);
  load_row_frags<T, D>(dO + base, my_q, S, h, rs, dof);

  // D = rowsum(dO * O) in float, from the O the forward produced.
  float dpart = 0.f;
  {
    typename M::frag of[KS_D];
    load_row_frags<T, D>(O + base, my_q, S, h, rs, of);
#pragma unroll
    for (int ks = 0; ks < KS_D; ++ks) {
      if constexpr (M::KL == 1) {
        dpart = fmaf((float)dof[ks], (float)of[ks], dpart);
      } else {
#pragma unroll
        for (int i = 0; i < M::KL; ++i) dpart = fmaf((float)dof[ks][i], (float)of[ks][i], dpart);
      }
    }
  }
  const float Dq = halves_sum(dpart);
  const float lse = my_q < S ? LSE[(int64_t)bh * S + my_q] : 0.f;
  const float lse2 = lse * kLog2e;
  const int Sp = ws_rows(S);
  if (h == 0 && my_q < Sp) {  // workspace of this head: D row, then -LSE/scale row; padding entries are zero
    float* wsh = Dvec + (int64_t)bh * 2 * Sp;
    wsh[my_q] = my_q < S ? Dq : 0.f;
    wsh[Sp + my_q] = my_q < S ? -lse / scale : 0.f;
  }

  const int kend = CAUSAL ? min(S, q0 + BQ) : S;
  const int n_kt = (kend + BK - 1) / BK;
  f32x16 dqacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) dqacc[dt] = f32x16{};

  TileStage<T, D, BK, NT> sk, sv;
  sk.load(Kb, 0, S, tid, rs);
  sv.load(Vb, 0, S, tid, rs);
  sk.store(smem, tid);
  sv.store(smem + TILE, tid);
  __syncthreads();

  for (int kt = 0; kt < n_kt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < n_kt) {
      sk.load(Kb, (kt + 1) * BK, S, tid, rs);
      sv.load(Vb, (kt + 1) * BK, S, tid, rs);
    }
    const char* lk = smem + buf * 2 * TILE;
    const char* lv = lk + TILE;
#pragma unroll
    for (int sb = 0; sb < BK / 32; ++sb) {
      const int k0 = kt * BK + sb * 32;
      if (k0 >= kend || (CAUSAL && k0 > qw + 31)) continue;  // wave-uniform skip
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS_D; ++ks) {
        s = M::run(read_row_frag<T, D>(lk, sb * 32 + r, ks, h), qf[ks], s);
        dp = M::run(read_row_frag<T, D>(lv, sb * 32 + r, ks, h), dof[ks], dp);
      }
      if ((CAUSAL && k0 + 31 > qw) || k0 + 32 > S) {
        // masked scores get the finite sentinel, whose exponential is exactly 0
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int key = k0 + acc_row(a, h);
          if (key >= S || (CAUSAL && key > my_q)) s[a] = kMasked;
        }
      }
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        const float p = exp2_hw(fmaf(s[a], c, -lse2));
        dp[a] = p * (dp[a] - Dq);  // dS^T
      }
#pragma unroll
      for (int ks = 0; ks < KS_32; ++ks) {
        const typename M::frag db = M::pack(dp, ks);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          dqacc[dt] = M::run(TransRead<T, D>::read(lk, sb * 32, ks, dt * 32, lane), db, dqacc[dt]);
      }
    }
    if (kt + 1 < n_kt) {
      sk.store(smem + (buf ^ 1) * 2 * TILE, tid);
      sv.store(smem + (buf ^ 1) * 2 * TILE + TILE, tid);
    }
    __syncthreads();
  }

  if (my_q < S) {
    T* row = dQ + base + (int64_t)my_q * rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<T>(row + dt * 32 + 8 * g + 4 * h, dqacc[dt][4 * g] * scale, dqacc[dt][4 * g + 1] * scale,
                  dqacc[dt][4 * g + 2] * scale, dqacc[dt][4 * g + 3] * scale);
  }
}

template <typename T, int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(const T* __restrict__ Q, const T* __restrict__ K,
                                                            const T* __restrict__ V, const T* __restrict__ dO,
                                                            const float* __restrict__ LSE,
                                                            const float* __restrict__ Dvec, T* __restrict__ dK,
                                                            T* __restrict__ dV, int S, int BH, int n_ktiles,
                                                            float c, float scale, int H, int seq_major) {
  typedef Mma<T> M;
  constexpr int BKV = 128, BQ = 64, NT = 256;
  constexpr int KS_D = D / M::K, KS_32 = 32 / M::K, DT = D / 32;
  constexpr int TILE = BQ * D * (int)sizeof(T);
  constexpr int VEC = BQ * 4;                 // one float per query row
  constexpr int BUF = 2 * TILE + 2 * VEC;     // Q, dO, LSE*log2e, D
  __shared__ __attribute__((aligned(16))) char smem[2 * BUF];

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, kt;
  tile_of_block(blockIdx.x, BH, n_ktiles, false, bh, kt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const T* Qb = Q + base;
  const T* dOb = dO + base;
  const float* Lb = LSE + (int64_t)bh * S;
  const float* Db = Dvec + (int64_t)bh * 2 * ws_rows(S);

  const int k0 = kt * BKV, kw = k0 + 32 * w, my_k = kw + r;
  typename M::frag kf[KS_D], vf[KS_D];
  load_row_frags<T, D>(K + base, my_k, S, h, rs, kf);
  load_row_frags<T, D>(V + base, my_k, S, h, rs, vf);

  const int qstart = CAUSAL ? k0 : 0;  // causal: the query loop starts at the diagonal
  const int qt0 = qstart / BQ;
  const int n_qt = (S + BQ - 1) / BQ;
  f32x16 dkacc[DT], dvacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    dkacc[dt] = f32x16{};
    dvacc[dt] = f32x16{};
  }

  TileStage<T, D, BQ, NT> sq, sdo;
  float vec = 0.f;  // threads 0..63 stage LSE*log2e, threads 64..127 stage D
  auto load_tile = [&](int qt) {
    sq.load(Qb, qt * BQ, S, tid, rs);
    sdo.load(dOb, qt * BQ, S, tid, rs);
    const int row = qt * BQ + (tid & 63);
    vec = 0.f;
    if (tid < 64) {
      if (row < S) vec = Lb[row] * kLog2e;
    } else if (tid < 128) {
      if (row < S) vec = Db[row];
    }
  };
  auto store_tile = [&](char* b) {
    sq.store(b, tid);
    sdo.store(b + TILE, tid);
    if (tid < 128) ((float*)(b + 2 * TILE))[tid] = vec;  // [0,64): LSE*log2e, [64,128): D
  };

  if (qt0 < n_qt) {
    load_tile(qt0);
    store_tile(smem);
  }
  __syncthreads();

  for (int qt = qt0; qt < n_qt; ++qt) {
    const int buf = (qt - qt0) & 1;
    if (qt + 1 < n_qt) load_tile(qt + 1);
    const char* lq = smem + buf * BUF;
    const char* ldo = lq + TILE;
    const float* llse = (const float*)(lq + 2 * TILE);
    const float* ld = llse + BQ;
#pragma unroll
    for (int sb = 0; sb < BQ / 32; ++sb) {
      const int q0 = qt * BQ + sb * 32;
      if (q0 >= S || (CAUSAL && q0 + 31 < kw)) continue;  // wave-uniform skip
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS_D; ++ks) {
        s = M::run(read_row_frag<T, D>(lq, sb * 32 + r, ks, h), kf[ks], s);
        dp = M::run(read_row_frag<T, D>(ldo, sb * 32 + r, ks, h), vf[ks], dp);
      }
      // s[a], dp[a]: query q0 + acc_row(a, h), key my_k
      if ((CAUSAL && q0 < kw + 31) || q0 + 32 > S) {
        // masked scores get the finite sentinel, whose exponential is exactly 0
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int qry = q0 + acc_row(a, h);
          if (qry >= S || (CAUSAL && my_k > qry)) s[a] = kMasked;
        }
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l4 = *(const f32x4*)(llse + sb * 32 + 8 * g + 4 * h);
        const f32x4 d4 = *(const f32x4*)(ld + sb * 32 + 8 * g + 4 * h);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int a = 4 * g + j;
          const float p = exp2_hw(fmaf(s[a], c, -l4[j]));
          s[a] = p;
          dp[a] = p * (dp[a] - d4[j]);  // dS
        }
      }
#pragma unroll
      for (int ks = 0; ks < KS_32; ++ks) {
        const typename M::frag pb = M::pack(s, ks);
        const typename M::frag db = M::pack(dp, ks);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          dvacc[dt] = M::run(TransRead<T, D>::read(ldo, sb * 32, ks, dt * 32, lane), pb, dvacc[dt]);
          dkacc[dt] = M::run(TransRead<T, D>::read(lq, sb * 32, ks, dt * 32, lane), db, dkacc[dt]);
        }
      }
    }
    if (qt + 1 < n_qt) store_tile(smem + (buf ^ 1) * BUF);
    __syncthreads();
  }

  if (my_k < S) {
    T* krow = dK + base + (int64_t)my_k * rs;
    T* vrow = dV + base + (int64_t)my_k * rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = dt * 32 + 8 * g + 4 * h;
        store4<T>(krow + col, dkacc[dt][4 * g] * scale, dkacc[dt][4 * g + 1] * scale, dkacc[dt][4 * g + 2] * scale,
                  dkacc[dt][4 * g + 3] * scale);
        store4<T>(vrow + col, dvacc[dt][4 * g], dvacc[dt][4 * g + 1], dvacc[dt][4 * g + 2], dvacc[dt][4 * g + 3]);
      }
  }
}

template <typename T, int D, bool CAUSAL>
static hipError_t launch_bwd_t(const BwdArgs& a, int phase, hipStream_t st) {
  const float c = a.scale * kLog2e;
  if (phase != 2) {
    const int n_qtiles = (a.S + 127) / 128;
    hipLaunchKernelGGL((attn_bwd_dq_kernel<T, D, CAUSAL>), dim3((unsigned)((int64_t)a.BH * n_qtiles)), dim3(256),
                       0, st, (const T*)a.q, (const T*)a.k, (const T*)a.v, (const T*)a.o, (const T*)a.dout, a.lse,
                       (T*)a.dq, a.ws, a.S, a.BH, n_qtiles, c, a.scale, a.H, (int)a.seq_major);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || phase == 1) return e;
  }
  const int n_ktiles = (a.S + 127) / 128;
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, D, CAUSAL>), dim3((unsigned)((int64_t)a.BH * n_ktiles)), dim3(256),
                     0, st, (const T*)a.q, (const T*)a.k, (const T*)a.v, (const T*)a.dout, a.lse, a.ws,
                     (T*)a.dk, (T*)a.dv, a.S, a.BH, n_ktiles, c, a.scale, a.H, (int)a.seq_major);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_bwd_d(const BwdArgs& a, int phase, hipStream_t st) {
  return a.causal ? launch_bwd_t<T, D, true>(a, phase, st) : launch_bwd_t<T, D, false>(a, phase, st);
}

hipError_t launch_bwd(const BwdArgs& a, int phase, hipStream_t st) {
  if (a.bf16) return launch_bwd_bf16(a, phase, st);
  return a.D == 64 ? launch_bwd_d<float, 64>(a, phase, st) : launch_bwd_d<float, 128>(a, phase, st);
}

// upper bound over the backward launch shapes (the smallest key tile is 64 rows)
int64_t bwd_grid_blocks(int BH, int S) { return (int64_t)BH * ((S + 63) / 64); }

}  // namespace cattn
