"""libgem: the GEM master-side commit pipeline on AMD MI355X (gfx950)."""
