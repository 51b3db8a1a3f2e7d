#!/bin/sh
# Builds the CPU oracle (plain C, float64, OpenMP). -ffp-contract=off keeps
# every multiply and add separately rounded so vector and scalar loop bodies
# give identical results.
set -e
cd "$(dirname "$0")"
gcc -O3 -mavx2 -mfma -ffp-contract=off -fno-math-errno -fopenmp -fPIC -shared -o liborc.so orc.c -lm
