"""CPU float64 oracle of the xHC connection.  Test infrastructure only."""
