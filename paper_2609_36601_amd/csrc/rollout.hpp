// Rollout kernels: student draft sampling and the first-rejection commit of a
// speculative wave (SAKI App. I, steps 1, 7 and 8; App. F).  Included by
// saki.hip inside namespace saki, after the verification kernel.
#pragma once

// ---------------------------------------------------------------------------
// Draft sampling, z ~ p = softmax(s), by the two-level exponential race on the
// proposal streams.  One workgroup per row: one read of the row for the chunk
// masses (each wave owns whole chunks, shifted by the chunk's own maximum, so
// no running maximum is needed: the race compares ln W_c, and a per-chunk
// shift is carried in the key), then the entry race inside the winning chunk
// re-reads one chunk.
// ---------------------------------------------------------------------------
struct SampleParams {
  const void* s;
  int64_t n_rows;
  int64_t stride;
  int64_t row_offset;
  int64_t row_step;
  int V;
  uint64_t seed;
  int32_t* token;
  uint8_t* status;
};

// Mass of one chunk from this lane's 16 entries s (valid mask vm): the chunk's
// maximum and the sum of 2^((s - max) log2 e) over the wave.
template <bool TAIL>
__device__ __forceinline__ bool chunk_mass(const float* s, uint32_t vm, float* ref, float* sum) {
  float m = -finf();
  bool fin = true;
#pragma unroll
  for (int e = 0; e < EPL; ++e)
    if (!TAIL || ((vm >> e) & 1u)) {
      m = fmaxf(m, s[e]);
      fin = fin && (s[e] - s[e] == 0.0f);  // false for NaN and +-inf
    }
  const float cm = wave_max(m);
  float acc = 0.0f;
#pragma unroll
  for (int e = 0; e < EPL; ++e)
    if (!TAIL || ((vm >> e) & 1u)) acc += fexp2((s[e] - cm) * LOG2E);
  *ref = cm;
  *sum = wave_sum(acc);
  return fin;
}

// One workgroup of SNT = 512 threads (eight waves) per row and one workgroup
// per CU: rollout batches are a few hundred rows, so a row's sweep is spread
// over more waves, each streaming its chunks with the next chunk's loads in
// flight (the row engine's chunk loop, on the one array).
constexpr int SAMPLE_NT = 512;

template <typename T>
__global__ __launch_bounds__(SAMPLE_NT, 1) void sample_kernel(SampleParams P) {
  constexpr int SNT = SAMPLE_NT;
  __shared__ RowShared<SNT> sh;
  Block<SNT> B(sh);
  constexpr int NW = SNT / WAVE;
  const int V = P.V;
  const int nch = (V + CHUNK - 1) / CHUNK;
  for (int64_t r = blockIdx.x; r < P.n_rows; r += gridDim.x) {
    const T* srow = static_cast<const T*>(P.s) + r * P.stride;
    const uint64_t g = static_cast<uint64_t>(P.row_offset + r * P.row_step);
    bool fin = true;
    for_chunks1<T, NW>(srow, V, B.wave, B.lane, [&](auto tail, const float* s, uint32_t vm, int c) {
      constexpr bool TAIL = decltype(tail)::value;
      float ref, sum;
      fin = chunk_mass<TAIL>(s, vm, &ref, &sum) && fin;
      if (B.lane == 0) {
        sh.chunk_a[c] = ref;
        sh.chunk_b[c] = sum;
      }
    });
    // the block max is also the barrier that publishes the chunk masses
    const bool finite = B.max(fin ? 0.0f : 1.0f) == 0.0f;
    int z = -1;
    if (finite) {
      const int c0 = chunk_race<SNT>(B, nch, P.seed, PROP_CHUNK, g, [&](int c) {
        return static_cast<double>(sh.chunk_a[c]) + log(static_cast<double>(sh.chunk_b[c]));
      });
      z = elem_race<SNT>(B, c0 < nch ? c0 : 0, V, P.seed, PROP_ELEM, g,
                         [&](int v) { return Loader<T>::load1(srow + v); });
      if (z >= V) z = -1;  // unreachable for finite rows: every chunk has a winner
    }
    if (B.tid == 0) {
      P.token[r] = z;
      if (P.status) P.status[r] = finite ? SAKI_ROW_OK : SAKI_ROW_NONFINITE;
    }
  }
}

// ---------------------------------------------------------------------------
// Commit of one speculative wave: for each running sequence, append the
// accepted drafts and the correction (the per-position token of the
// verification) to its trajectory, with the per-position metadata in token
// order, cut at max_len; update length and done.  One thread per sequence:
// the work is a few stores per committed token.
// ---------------------------------------------------------------------------
struct CommitParams {
  saki_traj tr;
  int k;
  int eos;
  const int32_t* accepted_len;
  const int32_t* correction;
  saki_couple_out pp;
  int32_t* n_commit;
};

__global__ __launch_bounds__(256) void commit_kernel(CommitParams P) {
  const int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (b >= P.tr.n_seq) return;
  const saki_traj& T = P.tr;
  int32_t m = 0;
  const int32_t len = T.length[b];
  if (T.done[b] == SAKI_SEQ_RUNNING) {
    if (len < 0 || len > T.max_len) {
      T.done[b] = SAKI_SEQ_STOPPED;
    } else {
      int32_t n = P.accepted_len[b];
      n = n < 0 ? 0 : (n > P.k ? P.k : n);
      const int32_t want = n + ((n < P.k && P.correction[b] >= 0) ? 1 : 0);
      const int64_t room = T.max_len - len;
      m = static_cast<int32_t>(want < room ? want : room);
      int32_t last = -1;
      for (int32_t j = 0; j < m; ++j) {
        const int64_t r = b * P.k + j;
        const int64_t o = b * T.max_len + len + j;
        const int32_t y = P.pp.token[r];
        T.tokens[o] = y;
        if (T.corrected) T.corrected[o] = (j == n) ? 1 : 0;
        if (T.lambda) T.lambda[o] = P.pp.lambda ? P.pp.lambda[r] : nanf_();
        if (T.kl) T.kl[o] = P.pp.kl ? P.pp.kl[r] : nanf_();
        if (T.tv) T.tv[o] = P.pp.tv ? P.pp.tv[r] : nanf_();
        if (T.logp_token) T.logp_token[o] = P.pp.logp_token ? P.pp.logp_token[r] : nanf_();
        if (T.logt_token) T.logt_token[o] = P.pp.logt_token ? P.pp.logt_token[r] : nanf_();
        if (T.teacher_argmax) T.teacher_argmax[o] = P.pp.teacher_argmax ? P.pp.teacher_argmax[r] : -1;
        last = y;
      }
      T.length[b] = len + m;
      if (m == 0)
        T.done[b] = SAKI_SEQ_STOPPED;
      else if (len + m >= T.max_len || (P.eos >= 0 && last == P.eos))
        T.done[b] = SAKI_SEQ_FINISHED;
    }
  }
  if (P.n_commit) P.n_commit[b] = m;
}
