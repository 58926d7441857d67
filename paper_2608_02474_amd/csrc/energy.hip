// Audio energy anchor (Sec. 3.3, "Cross-modal Saliency Anchors"): per-segment
// STFT power, pooled into mel-width bands and latent frames.
//
// Kernel 1 (energy_frames): one workgroup per (segment, STFT frame).  The
// windowed frame and a full-period twiddle table live in LDS in fp64; each
// thread evaluates whole one-sided bins k directly from the DFT sum, writes
// |X_k|^2 and the bin's band to LDS, and one thread per band sums its bins in
// ascending order.
// This runs once per clip on ~10^2-10^3 frames, so a direct O(n_fft^2) DFT in
// fp64 costs microseconds and keeps the result within fp64 rounding of the
// definition; an FFT would save nothing measurable here.
// Kernel 2 (energy_reduce): one workgroup sums the per-frame band energies of
// each segment in frame order, then forms e_t and e_t / max e.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace echo {

constexpr int kEnergyThreads = 256;   // energy_reduce (power of two: tree reduction)
constexpr int kFrameThreads = 512;    // energy_frames: one thread per one-sided bin up to n_fft 1022
constexpr int kMaxFft = 2048;

__device__ __forceinline__ int band_of_bin(int k, int n_fft, int sr, int n_bands) {
  const double mel_top = 2595.0 * log10(1.0 + (0.5 * sr) / 700.0);
  const double width = mel_top / n_bands;
  const double f = static_cast<double>(k) * sr / n_fft;
  const double m = 2595.0 * log10(1.0 + f / 700.0);
  int b = static_cast<int>(floor(m / width));
  return b < n_bands - 1 ? b : n_bands - 1;
}

__global__ void __launch_bounds__(kFrameThreads)
energy_frames(const float* __restrict__ audio, int64_t n_samples, int T, int n_fft, int hop,
              int n_bands, int sr, int max_frames, double* __restrict__ part) {
  extern __shared__ double lds[];
  double* xw = lds;                 // [n_fft] windowed frame
  double* tc = lds + n_fft;         // [n_fft] cos(2 pi m / n_fft)
  double* ts = lds + 2 * n_fft;     // [n_fft] sin(2 pi m / n_fft)
  double* pw = lds + 3 * n_fft;     // [n_fft/2 + 1] |X_k|^2
  int* bandof = reinterpret_cast<int*>(lds + 3 * n_fft + n_fft / 2 + 1);  // [n_fft/2 + 1] band of bin k
  const int t = blockIdx.y, f = blockIdx.x;
  const int64_t a = (static_cast<int64_t>(t) * n_samples) / T;
  const int64_t b = (static_cast<int64_t>(t + 1) * n_samples) / T;
  const int64_t len = b - a;
  const int nf = len < n_fft ? 1 : static_cast<int>(1 + (len - n_fft) / hop);
  double* out = part + (static_cast<int64_t>(t) * max_frames + f) * n_bands;
  if (f >= nf) {  // frame slot past this segment's frame count: contributes zero
    for (int i = threadIdx.x; i < n_bands; i += blockDim.x) out[i] = 0.0;
    return;
  }
  const int64_t start = a + static_cast<int64_t>(f) * hop;
  for (int n = threadIdx.x; n < n_fft; n += blockDim.x) {
    const double w = 0.5 - 0.5 * cospi(2.0 * n / n_fft);      // periodic Hann
    const int64_t s = start + n;
    const double v = (s < b) ? static_cast<double>(audio[s]) : 0.0;  // zero-pad short segments
    xw[n] = w * v;
    double sn, cs;
    sincospi(2.0 * n / n_fft, &sn, &cs);
    tc[n] = cs;
    ts[n] = sn;
  }
  __syncthreads();
  const int nbins = n_fft / 2 + 1;
  for (int k = threadIdx.x; k < nbins; k += blockDim.x) {
    double re = 0.0, im = 0.0;
    int m = 0;  // (k * n) mod n_fft, advanced incrementally
    for (int n = 0; n < n_fft; ++n) {
      re = fma(xw[n], tc[m], re);
      im = fma(-xw[n], ts[m], im);
      m += k;
      if (m >= n_fft) m -= n_fft;
    }
    pw[k] = re * re + im * im;
    bandof[k] = band_of_bin(k, n_fft, sr, n_bands);
  }
  __syncthreads();
  for (int band = threadIdx.x; band < n_bands; band += blockDim.x) {
    double acc = 0.0;  // bins of the band in ascending order
    for (int k = 0; k < nbins; ++k)
      if (bandof[k] == band) acc += pw[k];
    out[band] = acc;
  }
}

__global__ void __launch_bounds__(kEnergyThreads)
energy_reduce(const double* __restrict__ part, int T, int max_frames, int n_bands,
              float* __restrict__ band_energy, float* __restrict__ frame_energy,
              float* __restrict__ frame_weight, double* __restrict__ e_scratch) {
  __shared__ double red[kEnergyThreads];
  double local_max = 0.0;
  for (int t = threadIdx.x; t < T; t += blockDim.x) {
    double tot = 0.0;
    for (int band = 0; band < n_bands; ++band) {
      double acc = 0.0;
      for (int f = 0; f < max_frames; ++f)
        acc += part[(static_cast<int64_t>(t) * max_frames + f) * n_bands + band];
      band_energy[static_cast<int64_t>(t) * n_bands + band] = static_cast<float>(acc);
      tot += acc;
    }
    const double e = sqrt(tot);
    e_scratch[t] = e;
    frame_energy[t] = static_cast<float>(e);
    local_max = fmax(local_max, e);
  }
  red[threadIdx.x] = local_max;
  __syncthreads();
  for (int s = blockDim.x / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + s]);
    __syncthreads();
  }
  const double mx = red[0];
  for (int t = threadIdx.x; t < T; t += blockDim.x)
    frame_weight[t] = mx > 0.0 ? static_cast<float>(e_scratch[t] / mx) : 1.0f;
}

int energy_max_frames(int64_t n_samples, int T, int n_fft, int hop) {
  // the longest segment has ceil(n / T) samples
  const int64_t longest = (n_samples + T - 1) / T;
  return longest < n_fft ? 1 : static_cast<int>(1 + (longest - n_fft) / hop);
}

hipError_t launch_energy(const float* audio, int64_t n_samples, int T, int sr, int n_fft, int hop,
                         int n_bands, float* band_energy, float* frame_energy, float* frame_weight,
                         double* part, double* e_scratch, hipStream_t stream) {
  const int mf = energy_max_frames(n_samples, T, n_fft, hop);
  const size_t lds = sizeof(double) * (3 * n_fft + n_fft / 2 + 1) + sizeof(int) * (n_fft / 2 + 1);
  hipError_t e = ECHO_LAUNCH("energy_frames", energy_frames, dim3(mf, T), dim3(kFrameThreads), lds,
                             stream, audio, n_samples, T, n_fft, hop, n_bands, sr, mf, part);
  if (e != hipSuccess) return e;
  return ECHO_LAUNCH("energy_reduce", energy_reduce, dim3(1), dim3(kEnergyThreads), 0, stream, part, T,
                     mf, n_bands, band_energy, frame_energy, frame_weight, e_scratch);
}

}  // namespace echo
