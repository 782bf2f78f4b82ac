"""Plain CPU oracle of the MosaicKV hot path.  Test infrastructure only."""
