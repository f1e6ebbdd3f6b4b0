"""MI355X-native in-place real-domain FFT (rdFFT) and block-circulant layer."""
