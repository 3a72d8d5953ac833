# Build without Python: the HIP library for gfx950 (and its two measurement builds) and the fp64
# oracle, with the same flags as paper_2510_13223_amd/build.py and oracle.build().
#
#   make            libbana.so and liboracle.so
#   make variants   libbana_racecheck.so (BANA_LDS_RACE_CHECK) and libbana_timeline.so (BANA_WAVE_TIMELINE)
#   make clean

HIPCC ?= hipcc
CC ?= gcc
ARCH ?= gfx950
PKG := paper_2510_13223_amd
CSRC := $(PKG)/csrc
SRCS := attn_partial.hip merge.hip migrate.hip validate.hip debug_rows.hip gather_read.hip scratch.hip bana_api.cpp
HDRS := include/bana.h $(wildcard $(CSRC)/*.h)
HIPFLAGS := --offload-arch=$(ARCH) -O3 -fPIC -std=c++17 -Wall -Xclang -target-feature -Xclang -packed-fp32-ops \
            -Iinclude -I$(CSRC)
OBJ := _build/make

all: $(PKG)/libbana.so oracle/liboracle.so
variants: $(PKG)/libbana_racecheck.so $(PKG)/libbana_timeline.so

# $(1): object folder, $(2): extra flags, $(3): library
define hip_library
$(OBJ)/$(1)/%.o: $(CSRC)/% $(HDRS)
	@mkdir -p $$(@D)
	$$(HIPCC) $$(HIPFLAGS) $(2) -x hip -c $$< -o $$@
$(3): $(addprefix $(OBJ)/$(1)/,$(addsuffix .o,$(SRCS)))
	$$(HIPCC) --offload-arch=$$(ARCH) -shared -fPIC $$^ -o $$@
endef

$(eval $(call hip_library,product,,$(PKG)/libbana.so))
$(eval $(call hip_library,racecheck,-DBANA_LDS_RACE_CHECK,$(PKG)/libbana_racecheck.so))
$(eval $(call hip_library,timeline,-DBANA_WAVE_TIMELINE,$(PKG)/libbana_timeline.so))

oracle/liboracle.so: oracle/oracle.c
	$(CC) -O2 -std=c11 -fopenmp -fPIC -shared $< -o $@ -lm

clean:
	rm -rf $(OBJ) $(PKG)/libbana.so $(PKG)/libbana_racecheck.so $(PKG)/libbana_timeline.so oracle/liboracle.so

.PHONY: all variants clean
