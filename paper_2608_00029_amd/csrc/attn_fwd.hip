// Fused causal attention forward for gfx950 (section 4.2 of the Nova paper).
//
// One workgroup of 4 waves owns a tile of 128 queries of one (batch, head);
// each wave owns 32 consecutive queries.  Key/value tiles of 64 rows are
// staged HBM -> registers -> LDS with double buffering, so the global loads of
// tile t+1 are in flight while tile t is consumed.  Per 32-key block the wave
// computes the TRANSPOSED score block S^T = K Q^T on the matrix cores, so that
// each lane holds 16 keys of ONE query: the row max and row sum are in-lane
// reductions plus a single cross-half exchange.  The online softmax runs in
// base 2 with scale*log2(e) folded into one fused multiply-add, the causal
// mask is applied only on blocks that straddle the diagonal (or the ragged
// end of the sequence), blocks entirely above the diagonal are never visited
// (loop clamping), and the probabilities feed O^T += V^T P^T directly from
// registers.  S and P never touch LDS or HBM; 1/l is applied once in the
// epilogue, where LSE = ln2 * (max*scale*log2e + log2 l) is also written.
#include "attn_device.h"
#include "attn_launch.h"

namespace cattn {

template <typename T, int D, bool CAUSAL>
__global__ __launch_bounds__(256) void attn_fwd_kernel(const T* __restrict__ Q, const T* __restrict__ K,
                                                       const T* __restrict__ V, T* __restrict__ O,
                                                       float* __restrict__ LSE, int S, int BH, int n_qtiles,
                                                       float c, int H, int seq_major) {
  typedef Mma<T> M;
  constexpr int BQ = 128, BK = 64, NT = 256;
  constexpr int KS_D = D / M::K;      // k-steps over the head dimension
  constexpr int KS_32 = 32 / M::K;    // k-steps over a 32-row block
  constexpr int DT = D / 32;          // 32-wide column blocks of the output
  constexpr int TILE = BK * D * (int)sizeof(T);
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * TILE];  // [buffer][K, V]

  const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in an SGPR
  int bh, qt;
  tile_of_block(blockIdx.x, BH, n_qtiles, CAUSAL, bh, qt);
  const Rows rw = rows_of(bh, H, S, D, seq_major);
  const int64_t base = rw.base;
  const int rs = rw.rs;
  const T* Qb = Q + base;
  const T* Kb = K + base;
  const T* Vb = V + base;

  const int q0 = qt * BQ, qw = q0 + 32 * w, my_q = qw + r;
  typename M::frag qf[KS_D];
  load_row_frags<T, D>(Qb, my_q, S, h, rs, qf);

  const int kend = CAUSAL ? min(S, q0 + BQ) : S;  // causal loop clamping
  const int n_kt = (kend + BK - 1) / BK;

  float m = kMasked;   // running softmax offset, in raw-score units (scale folded in later)
  float lsum = 0.f;    // running sum of this half's probabilities
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};

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
      f32x16 s = f32x16{};
#pragma unroll
      for (int ks = 0; ks < KS_D; ++ks) s = M::run(read_row_frag<T, D>(lk, sb * 32 + r, ks, h), qf[ks], s);
      // s[a] = raw score of key k0 + acc_row(a, h) against query my_q
      if ((CAUSAL && k0 + 31 > qw) || k0 + 32 > S) {
#pragma unroll
        for (int a = 0; a < 16; ++a) {
          const int key = k0 + acc_row(a, h);
          if (key >= S || (CAUSAL && key > my_q)) s[a] = kMasked;
        }
      }
      float mx = s[0];
#pragma unroll
      for (int a = 1; a < 16; ++a) mx = fmaxf(mx, s[a]);
      mx = halves_max(mx);
      // Lazy rescaling: the running offset m only moves when the block's max
      // exceeds it by more than 2^kRescaleLog2 in probability units, so P stays
      // <= 2^kRescaleLog2 and the O/l rescale (a multiply of every accumulator)
      // is skipped in almost every block.  O/l and LSE are exact for any m.
      const bool grow = (mx - m) * c > kRescaleLog2;
      if (__builtin_amdgcn_ballot_w64(grow)) {  // wave-uniform branch
        const float m_new = grow ? mx : m;
        const float alpha = exp2_hw((m - m_new) * c);
        m = m_new;
        lsum *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
      }
      const float mc = m * c;
      float psum = 0.f;
#pragma unroll
      for (int a = 0; a < 16; ++a) {
        s[a] = exp2_hw(fmaf(s[a], c, -mc));
        psum += s[a];
      }
      lsum += psum;
#pragma unroll
      for (int ks = 0; ks < KS_32; ++ks) {
        const typename M::frag pb = M::pack(s, ks);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          oacc[dt] = M::run(TransRead<T, D>::read(lv, sb * 32, ks, dt * 32, lane), pb, oacc[dt]);
      }
    }
    if (kt + 1 < n_kt) {
      // buffer buf^1 was last read in iteration kt-1, which every wave finished
      // before the barrier that closed it.
      sk.store(smem + (buf ^ 1) * 2 * TILE, tid);
      sv.store(smem + (buf ^ 1) * 2 * TILE + TILE, tid);
    }
    __syncthreads();
  }

  const float l = halves_sum(lsum);
  if (my_q < S) {
    const float inv = 1.0f / l;
    T* orow = O + base + (int64_t)my_q * rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        store4<T>(orow + dt * 32 + 8 * g + 4 * h, oacc[dt][4 * g] * inv, oacc[dt][4 * g + 1] * inv,
                  oacc[dt][4 * g + 2] * inv, oacc[dt][4 * g + 3] * inv);
    if (h == 0) LSE[(int64_t)bh * S + my_q] = (m * c + log2f(l)) * kLn2;
  }
}

template <typename T, int D, bool CAUSAL>
hipError_t launch_fwd_t(const FwdArgs& a, hipStream_t st) {
  const int n_qtiles = (a.S + 127) / 128;
  const int64_t blocks = (int64_t)a.BH * n_qtiles;
  hipLaunchKernelGGL((attn_fwd_kernel<T, D, CAUSAL>), dim3((unsigned)blocks), dim3(256), 0, st,
                     (const T*)a.q, (const T*)a.k, (const T*)a.v, (T*)a.o, a.lse, a.S, a.BH, n_qtiles,
                     a.scale * kLog2e, a.H, (int)a.seq_major);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_fwd_d(const FwdArgs& a, hipStream_t st) {
  return a.causal ? launch_fwd_t<T, D, true>(a, st) : launch_fwd_t<T, D, false>(a, st);
}

hipError_t launch_fwd(const FwdArgs& a, hipStream_t st) {
  if (a.bf16) return launch_fwd_bf16(a, st);
  return a.D == 64 ? launch_fwd_d<float, 64>(a, st) : launch_fwd_d<float, 128>(a, st);
}

// upper bound over the forward launch shapes (the smallest query tile is 32 rows)
int64_t fwd_grid_blocks(int BH, int S) { return (int64_t)BH * ((S + 31) / 32); }

}  // namespace cattn
