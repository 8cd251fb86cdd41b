"""CPU oracle of the rasterizer (test infrastructure only; see gs_oracle.h)."""
