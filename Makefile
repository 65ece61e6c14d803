# Builds the three shared libraries in-tree:
#   paper_2609_18178_amd/libpactshard.so  the gfx950 library (HIP kernels + C ABI)
#   oracle/liboracle.so                   the CPU oracle (test infrastructure)
#   workloads/libgen.so                   the seeded input generator
# `make -B` rebuilds everything.

HIPCC    ?= /opt/rocm/bin/hipcc
CC       ?= gcc
ARCH     ?= gfx950

PKG      := paper_2609_18178_amd
LIB      := $(PKG)/libpactshard.so
LIB_SRCS := $(wildcard $(PKG)/csrc/*.hip) $(wildcard $(PKG)/csrc/*.cpp)
LIB_HDRS := include/pactshard.h $(wildcard $(PKG)/csrc/*.h)

# Exact binary32: no contraction into FMA, correctly rounded '/' and sqrt,
# fp32 denormals kept; packed-fp32 instructions disabled for the device code.
HIPFLAGS := --offload-arch=$(ARCH) -O3 -std=c++17 -fPIC -shared \
            -ffp-contract=off -fno-fast-math -fhip-fp32-correctly-rounded-divide-sqrt \
            -fno-gpu-flush-denormals-to-zero \
            -Xclang -target-feature -Xclang -packed-fp32-ops \
            -Wall -Wno-unused-command-line-argument -Iinclude

ORACLE_FLAGS := -O2 -std=c11 -ffp-contract=off -fno-fast-math -fno-math-errno \
                -fexcess-precision=standard -fPIC -shared -Wall -Wextra
GEN_FLAGS    := -O3 -std=c11 -fopenmp -fPIC -shared -Wall -Wextra

# A plain C caller of the library (test infrastructure: it links the oracle
# to check what the library computes); finds the in-tree libraries by rpath.
C_CALLER := tests/native/c_caller
ROCM     ?= /opt/rocm

all: oracle/liboracle.so workloads/libgen.so $(if $(LIB_SRCS),$(LIB) $(C_CALLER),)

oracle/liboracle.so: oracle/oracle.c oracle/oracle.h
	$(CC) $(ORACLE_FLAGS) -o $@ oracle/oracle.c -lm

workloads/libgen.so: workloads/gen.c
	$(CC) $(GEN_FLAGS) -o $@ workloads/gen.c

$(LIB): $(LIB_SRCS) $(LIB_HDRS)
	$(HIPCC) $(HIPFLAGS) -o $@ $(LIB_SRCS)

$(C_CALLER): tests/native/c_caller.c include/pactshard.h oracle/oracle.h $(LIB) oracle/liboracle.so workloads/libgen.so
	$(CC) -std=c99 -O2 -Wall -Wextra -D__HIP_PLATFORM_AMD__ -Iinclude -Ioracle -I$(ROCM)/include -o $@ $< \
	    -L$(PKG) -lpactshard -Loracle -loracle -Lworkloads -lgen -L$(ROCM)/lib -lamdhip64 \
	    -Wl,-rpath,'$$ORIGIN/../../$(PKG)' -Wl,-rpath,'$$ORIGIN/../../oracle' -Wl,-rpath,'$$ORIGIN/../../workloads' \
	    -Wl,-rpath,$(ROCM)/lib

# gfx950 assembly of the kernels, for inspection and the hazard test
isa: _build/kernels-gfx950.s
_build/kernels-gfx950.s: $(PKG)/csrc/kernels.hip $(LIB_HDRS)
	mkdir -p _build
	$(HIPCC) $(filter-out -shared -fPIC,$(HIPFLAGS)) --cuda-device-only -S -o $@ $(PKG)/csrc/kernels.hip

clean:
	rm -f $(LIB) oracle/liboracle.so workloads/libgen.so $(C_CALLER)
	rm -rf _build

.PHONY: all clean isa
