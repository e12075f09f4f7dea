"""fp64 CPU oracle of the DFlare draft step -- test infrastructure only."""
