#!/bin/sh
# Builds the CPU oracle's shared library (test infrastructure; never linked by the product).
set -e
cd "$(dirname "$0")"
gcc -O2 -fopenmp -fPIC -shared -std=c11 -Wall -Wextra -o libbc_oracle.so bc_oracle.c -lm
