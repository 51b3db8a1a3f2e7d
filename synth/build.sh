#!/bin/sh
# Builds the seeded-input generator (plain C, OpenMP).
set -e
cd "$(dirname "$0")"
gcc -O3 -mavx2 -mfma -fno-math-errno -fopenmp -fPIC -shared -o libsynth.so synth.c -lm
